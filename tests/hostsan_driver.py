"""Drives the host-side logic of a sanitizer build of the library (ASan + UBSan on the host code,
no GPU needed): size queries over many configurations, every argument check that returns before a
device call, NULL-context paths and error texts.  Run by tests/test_abi_cpu.py in a subprocess with
the sanitizer runtime preloaded; prints OK when every call returned the expected status."""
import ctypes
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2403_18647_amd import binding as B  # noqa: E402
from paper_2403_18647_amd import synth  # noqa: E402


def main(path):
    B.LIB_PATH = path
    L = B.lib()
    n = 0
    # size queries: valid shapes of every kind, and invalid ones
    for shape in (synth.TINY, synth.LLAMA7B, synth.LLAMA13B, synth.small_shape(d_ffn=690, vocab=7)):
        for mb, mc, mq in ((1, 1, 1), (1, 100, 6), (4, 1324, 1024), (8, 16427, 11), (3, 33, 4096)):
            cfg = B.make_config(shape, max_batch=mb, max_ctx=mc, max_block=mq)
            size = ctypes.c_size_t(0)
            rc = L.sdsat_query_sizes(ctypes.byref(cfg), ctypes.byref(size))
            assert rc in (0, -5), rc
            assert rc != 0 or size.value > 0
            n += 1
    bad = B.make_config(synth.TINY, max_batch=1, max_ctx=64, max_block=6)
    for field, value in (("head_dim", 96), ("max_block", 4097), ("d_model", 250), ("dtype", 7), ("n_layers", 0),
                         ("max_ctx", 0), ("vocab", 1), ("n_adaptive", -1), ("rms_eps", -1.0), ("rope_base", 0.0)):
        c = B.make_config(synth.TINY, max_batch=1, max_ctx=64, max_block=6)
        setattr(c, field, value)
        size = ctypes.c_size_t(0)
        assert L.sdsat_query_sizes(ctypes.byref(c), ctypes.byref(size)) < 0, field
        assert len(L.sdsat_last_error(None)) > 0
        n += 1
    assert L.sdsat_query_sizes(None, None) == -1
    assert L.sdsat_query_sizes(ctypes.byref(bad), None) == -1
    # init argument checks (all before any device call)
    out = ctypes.c_void_p(0)
    nw = 1 + 9 * synth.TINY.n_layers + 2
    ptrs = (ctypes.c_void_p * nw)(*([4096] * nw))
    assert L.sdsat_init(ctypes.byref(bad), ptrs, nw, ctypes.c_void_p(4096), 1 << 40, None, None) == -1
    assert L.sdsat_init(None, ptrs, nw, ctypes.c_void_p(4096), 1 << 40, None, ctypes.byref(out)) == -1
    assert L.sdsat_init(ctypes.byref(bad), ptrs, nw - 1, ctypes.c_void_p(4096), 1 << 40, None, ctypes.byref(out)) == -1
    assert L.sdsat_init(ctypes.byref(bad), ptrs, nw, ctypes.c_void_p(4097), 1 << 40, None, ctypes.byref(out)) == -1
    assert L.sdsat_init(ctypes.byref(bad), ptrs, nw, ctypes.c_void_p(4096), 16, None, ctypes.byref(out)) == -2
    nulls = (ctypes.c_void_p * nw)(*([4096] * (nw - 1) + [0]))
    assert L.sdsat_init(ctypes.byref(bad), nulls, nw, ctypes.c_void_p(4096), 1 << 40, None, ctypes.byref(out)) == -1
    assert out.value is None
    n += 6
    # every context call with a NULL context
    for name, args in (("sdsat_reset", (None, 1)), ("sdsat_set_cache_len", (None, 1, None)),
                       ("sdsat_forward_block", (None, 1, 1, None, None, None)),
                       ("sdsat_verify_greedy", (None, 1, 1, None, None, None, None)),
                       ("sdsat_verify_nucleus", (None, 1, 1, None, None, 1.0, 0.9, 0, 1, None, None, None)),
                       ("sdsat_commit_kv", (None, 1, 1, None, None)),
                       ("sdsat_generate", (None, 1, None, 1, 1, 0, None, 0, 0.0, 1.0, 0, 0, None, None)),
                       ("sdsat_kv_write", (None, 0, 1, 1, None, None, None)),
                       ("sdsat_attention", (None, 0, 1, 1, None, None, None)),
                       ("sdsat_profile_kernel", (None, 1, 1))):
        assert getattr(L, name)(*args) == -1, name
        n += 1
    assert L.sdsat_destroy(None) == 0 and L.sdsat_cache_len_ptr(None) is None
    # linear entry points: sizes and argument checks
    assert L.sdsat_linear_packed_bytes(1, 16, 32) == 16 * 32 * 2 and L.sdsat_linear_packed_bytes(1, 0, 32) == 0
    assert L.sdsat_linear_scratch_bytes(65, 16, 32) == 0
    p = ctypes.c_void_p(4096)
    assert L.sdsat_linear(2, 4, 16, 32, p, p, p, p, None) == -1
    assert L.sdsat_linear(1, 65, 16, 32, p, p, p, p, None) == -1
    assert L.sdsat_linear(1, 4, 16, 32, None, p, p, p, None) == -1
    assert L.sdsat_linear_pack(1, 16, 32, None, p, None) == -1
    assert L.sdsat_linear_noalloc(1, 4, 16, 32, None, p, p, None) == -1
    assert L.sdsat_linear_noalloc(0, 64, 16, 16416, p, p, p, None) == -1     # past the static scratch
    assert b"4 MiB" in L.sdsat_last_error(None)
    assert L.sdsat_stream_read(None, 16, None) == -1 and L.sdsat_stream_read(p, 24, None) == -1
    cnt = ctypes.c_int64(0)
    assert L.sdsat_kernel_samples(None, None, 0, ctypes.byref(cnt)) == -1
    n += 12
    print(f"OK {n} checks")


if __name__ == "__main__":
    main(sys.argv[1])
