"""Mutation sweep of the oracle's CPU pins (run by hand: python tests/mutation_sweep.py [names]).

Each entry plants one plausible mistake in a scratch copy of oracle/ (a dropped bf16 rounding, a
wrong sign, index, scale or tie rule, a transposed role) and runs tests/test_oracle_model.py and
tests/test_oracle_decode.py against the copy; every mutation must make at least one pin fail.  The
repository itself is never modified.  Prints one line per mutation and exits non-zero if any
mutation passes every pin."""
import os, shutil, subprocess, sys, tempfile
SRC = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MUTS = [
 ('oracle/model.py', 'rms_eps', 'x / np.sqrt(ms + eps) * gain', 'x / (np.sqrt(ms) + eps) * gain'),
 ('oracle/model.py', 'rms_gain', 'return x / np.sqrt(ms + eps) * gain', 'return x / np.sqrt(ms + eps)'),
 ('oracle/model.py', 'rope_sign', '[a * c - b * s, a * s + b * c]', '[a * c + b * s, -a * s + b * c]'),
 ('oracle/model.py', 'rope_freq', '-2.0 * i / head_dim', '-1.0 * i / head_dim'),
 ('oracle/model.py', 'rope_on_v', 'vh = rnd(vh)', 'vh = rnd(apply_rope(vh, cos, sin))'),
 ('oracle/model.py', 'rope_q_missing', 'qh = apply_rope(qh, cos, sin)', 'qh = qh'),
 ('oracle/model.py', 'rope_pos_shift', 'cos, sin = rope_cos_sin(positions, Dh, shape.rope_base)', 'cos, sin = rope_cos_sin(positions + 1, Dh, shape.rope_base)'),
 ('oracle/model.py', 'rope_table_f32', 'return (np.cos(ang).astype(np.float32).astype(np.float64),\n            np.sin(ang).astype(np.float32).astype(np.float64))', 'return (np.cos(ang), np.sin(ang))'),
 ('oracle/model.py', 'scale', 'scale = 1.0 / np.sqrt(Dh)', 'scale = 1.0 / Dh'),
 ('oracle/model.py', 'causal_future', 'np.tril(np.ones((q, q), dtype=bool))', 'np.tril(np.ones((q, q), dtype=bool), 1)'),
 ('oracle/model.py', 'silu_sign', 'z / (1.0 + np.exp(-z))', 'z / (1.0 + np.exp(z))'),
 ('oracle/model.py', 'swiglu_swap', 'a = rnd(silu(g) * u)', 'a = rnd(silu(u) * g)'),
 ('oracle/model.py', 'attn_resid', 'x = x + _linear(o, weights[p + "wo"], per_row)', 'x = _linear(o, weights[p + "wo"], per_row)'),
 ('oracle/model.py', 'ffn_resid', 'x = x + _linear(a, weights[p + "w_down"], per_row)', 'x = _linear(a, weights[p + "w_down"], per_row)'),
 ('oracle/model.py', 'k_round', 'kh = rnd(apply_rope(kh, cos, sin))', 'kh = apply_rope(kh, cos, sin)'),
 ('oracle/model.py', 'v_round', 'vh = rnd(vh)', 'vh = vh'),
 ('oracle/model.py', 'attn_norm_round', 'h = rnd(rms_norm(x, weights[p + "attn_norm"], eps))', 'h = rms_norm(x, weights[p + "attn_norm"], eps)'),
 ('oracle/model.py', 'attn_out_round', 'o = rnd(o.reshape(q, d))', 'o = o.reshape(q, d)'),
 ('oracle/model.py', 'ffn_norm_round', 'h2 = rnd(rms_norm(x, weights[p + "ffn_norm"], eps))', 'h2 = rms_norm(x, weights[p + "ffn_norm"], eps)'),
 ('oracle/model.py', 'swiglu_round', 'a = rnd(silu(g) * u)', 'a = silu(g) * u'),
 ('oracle/model.py', 'final_round', 'hf = rnd(rms_norm(x, weights["final_norm"], eps))', 'hf = rms_norm(x, weights["final_norm"], eps)'),
 ('oracle/model.py', 'final_norm_weight', 'hf = rnd(rms_norm(x, weights["final_norm"], eps))', 'hf = rnd(rms_norm(x, weights[p + "ffn_norm"], eps))'),
 ('oracle/model.py', 'attn_norm_weight', 'h = rnd(rms_norm(x, weights[p + "attn_norm"], eps))', 'h = rnd(rms_norm(x, weights[p + "ffn_norm"], eps))'),
 ('oracle/model.py', 'bf16_half_up', 'r = np.round(scaled)', 'r = np.floor(scaled + 0.5)'),
 ('oracle/model.py', 'wk_for_wv', 'vh = _linear(h, weights[p + "wv"], per_row).reshape(q, H, Dh)', 'vh = _linear(h, weights[p + "wk"], per_row).reshape(q, H, Dh)'),
 ('oracle/decode.py', 'greedy_accept_index', '        if int(drafts[j - 1]) != int(o[j - 1]):', '        if int(drafts[j - 1]) != int(o[j]):'),
 ('oracle/decode.py', 'commit_count', 'cache.commit(kv, range(m + 1))', 'cache.commit(kv, range(m + 2))'),
 ('oracle/decode.py', 'draft1_sampling_rows', 'if drafts is None and j > 0:', 'if drafts is None and j > 1:'),
 ('oracle/decode.py', 'nucleus_accept_index', '        if int(drafts[j - 1]) != int(out[j - 1]):', '        if int(drafts[j - 1]) != int(out[j]):'),
 ('oracle/sampling.py', 'top_p_strict', 'ok = np.nonzero(S >= p * E)[0]', 'ok = np.nonzero(S > p * E)[0]'),
 ('oracle/sampling.py', 'top_k_ties_high', 'np.lexsort((np.arange(V), -z))', 'np.lexsort((-np.arange(V), -z))'),
 ('oracle/sampling.py', 'temperature_mul', '/ float(np.float32(temperature))', '* float(np.float32(temperature))'),
 ('oracle/sampling.py', 'nucleus_strict_tau', 'ids = np.nonzero(zk >= tau)[0]', 'ids = np.nonzero(zk > tau)[0]'),
 ('oracle/sampling.py', 'splitmix_gamma', '_GOLDEN_GAMMA = 0x9E3779B97F4A7C15', '_GOLDEN_GAMMA = 0x9E3779B97F4A7C17'),
 ('oracle/sampling.py', 'uniform_bits', '(splitmix64(seed & _MASK, c + 1) >> 11)', '(splitmix64(seed & _MASK, c) >> 11)'),
 ('oracle/sampling.py', 'argmax_ties_high', 'return int(np.argmax(row))', 'return int(len(row) - 1 - np.argmax(row[::-1]))'),
 ('oracle/sampling.py', 'no_max_subtract', 'e = np.where(kept, np.exp(zk - zmax), 0.0)', 'e = np.where(kept, np.exp(zk - zmax + 1.0), 0.0)'),
]
tmp = tempfile.mkdtemp(prefix='mut_')
for d in ('oracle', 'tests', 'paper_2403_18647_amd'):
    shutil.copytree(os.path.join(SRC, d), os.path.join(tmp, d), ignore=shutil.ignore_patterns('*.so', '_build', '*.hipfb', '__pycache__', 'csrc'))
for f in ('pytest.ini', 'conftest.py', 'setup.cfg', 'pyproject.toml'):
    if os.path.exists(os.path.join(SRC, f)): shutil.copy(os.path.join(SRC, f), tmp)
tests = ['tests/test_oracle_model.py', 'tests/test_oracle_decode.py']
def run():
    r = subprocess.run([sys.executable, '-m', 'pytest', '-q', '-x', '-p', 'no:cacheprovider', *tests, '-m', 'not gpu'],
                       capture_output=True, text=True, cwd=tmp)
    return r.returncode, (r.stdout.strip().splitlines() or [''])[-1]
rc, last = run()
print('baseline', rc, last, flush=True)
unpinned = []
sel = sys.argv[1].split(',') if len(sys.argv) > 1 else None
for f, name, a, b in MUTS:
    if sel and name not in sel: continue
    p = os.path.join(tmp, f)
    orig = open(p).read()
    assert orig.count(a) >= 1, (name, a)
    open(p, 'w').write(orig.replace(a, b, 1))
    rc, last = run()
    open(p, 'w').write(orig)
    print(f'{name:24s}', 'FAILS' if rc else 'PASSES (unpinned)', last, flush=True)
    if not rc: unpinned.append(name)
print('unpinned:', unpinned)
shutil.rmtree(tmp)
sys.exit(1 if unpinned else 0)
