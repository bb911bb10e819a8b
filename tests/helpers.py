"""Shared helpers for the GPU parity tests (device setup, reference roundings)."""
import numpy as np

from oracle import model as M
from paper_2403_18647_amd import binding as B
from paper_2403_18647_amd import synth


def bf16_round_f32(a):
    """float32 -> nearest bf16 (ties to even), returned as float32 (test-side input rounding)."""
    u = np.ascontiguousarray(a, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def make_ctx(wl, max_batch, max_ctx, max_block, device="cuda"):
    weights = synth.device_weights(wl, device)
    cfg = B.make_config(wl.shape, max_batch=max_batch, max_ctx=max_ctx, max_block=max_block)
    return B.Context(cfg, weights)


def oracle_weights(wl):
    return M.Weights(wl.shape, {n: synth.tensor(wl, n) for n in synth.tensor_names(wl.shape)})


def small_bf16(**kw):
    """A reduced bf16 decoder with 128-wide heads and ragged vocabulary / FFN tiles."""
    shape = synth.small_shape(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=688, vocab=1000,
                              n_adaptive=5, rope_base=1e6, dtype="bf16")
    base = dict(name="small_bf16", shape=shape, seed=7, batch=1, k=5, prompt_len=40, max_new=48,
                gain_std=0.1)
    base.update(kw)
    return synth.Workload(**base)
