"""Host-side checks of the C-ABI library (no GPU needed): it loads, exports
every function include/sdsat.h declares, and its host-only size queries and
argument checks behave."""
import ctypes
import os
import re

import pytest

from paper_2403_18647_amd import binding as B
from paper_2403_18647_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sdsat.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sdsat_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_boundary_calls():
    names = _declared()
    for n in ("sdsat_init", "sdsat_forward_block", "sdsat_verify_greedy", "sdsat_verify_nucleus",
              "sdsat_commit_kv", "sdsat_generate", "sdsat_destroy", "sdsat_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = B.lib()
    for n in _declared():
        assert hasattr(L, n), n
    assert set(_declared()) == set(B.EXPORTS)


def test_query_sizes_host_only():
    cfg = B.make_config(synth.TINY, max_batch=1, max_ctx=128, max_block=6)
    a = B.sdsat_query_sizes(cfg)
    cfg2 = B.make_config(synth.TINY, max_batch=1, max_ctx=1024, max_block=6)
    b = B.sdsat_query_sizes(cfg2)
    assert 0 < a < b
    # the KV cache grows by 2 (K, V) * layers * heads * head_dim * 4 bytes per extra slot
    per_slot = 2 * synth.TINY.n_layers * synth.TINY.d_model * 4
    assert b - a >= per_slot * (1024 - 128)
    big = B.sdsat_query_sizes(B.make_config(synth.LLAMA7B, max_batch=1, max_ctx=1024, max_block=6))
    weights = 32 * (4 * 4096 * 4096 + 3 * 4096 * 11008) * 2 + 32016 * 4096 * 2
    assert big > weights


@pytest.mark.parametrize("field,value,code", [("head_dim", 96, B.ERRORS and -5), ("max_block", 4097, -5),
                                              ("d_model", 250, -1), ("dtype", 7, -1), ("n_layers", 0, -1)])
def test_query_sizes_rejects_bad_configs(field, value, code):
    cfg = B.make_config(synth.TINY, max_batch=1, max_ctx=128, max_block=6)
    setattr(cfg, field, value)
    with pytest.raises(B.SdsatError) as e:
        B.sdsat_query_sizes(cfg)
    assert e.value.code == code


def test_linear_sizes():
    assert B.sdsat_linear_packed_bytes(1, 16, 32) == 16 * 32 * 2
    assert B.sdsat_linear_packed_bytes(0, 17, 33) == 32 * 64 * 4          # padded to 16 x 32 tiles
    assert B.sdsat_linear_scratch_bytes(65, 16, 32) == 0                  # M > 64 unsupported
    assert B.sdsat_linear_scratch_bytes(6, 4096, 4096) > 0


def test_null_context_is_rejected_without_touching_the_gpu():
    L = B.lib()
    assert L.sdsat_reset(None, 1) == -1
    assert L.sdsat_forward_block(None, 1, 1, None, None, None) == -1
    assert L.sdsat_destroy(None) == 0
    assert b"ctx" in L.sdsat_last_error(None)


def test_measurement_helpers_reject_bad_arguments_on_the_host():
    L = B.lib()
    n = ctypes.c_int64(0)
    assert L.sdsat_kernel_samples(None, None, 0, ctypes.byref(n)) == -1
    assert L.sdsat_stream_read(None, 16, None) == -1            # NULL source with bytes to read
    assert L.sdsat_stream_read(ctypes.c_void_p(4096), 24, None) == -1   # not a multiple of 16
    assert b"multiple of 16" in L.sdsat_last_error(None)


def test_host_runtime_under_address_and_undefined_behaviour_sanitizers():
    """The host runtime built with ASan + UBSan (libsdsat_hostsan.so, built with the library): size
    queries over many configurations, every argument check that returns before a device call, the
    NULL-context paths and error texts, driven in a process with the sanitizer runtime preloaded.
    Any heap overflow, use after free or undefined behaviour in those paths aborts the process."""
    import subprocess
    import sys
    lib = os.path.join(ROOT, "paper_2403_18647_amd", "libsdsat_hostsan.so")
    assert os.path.exists(lib), "libsdsat_hostsan.so is not built; run __graft_entry__.build()"
    rt = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    assert os.path.isabs(rt) and os.path.exists(rt), "no libasan to preload"
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "hostsan_driver.py"), lib], env=env,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "OK" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]
