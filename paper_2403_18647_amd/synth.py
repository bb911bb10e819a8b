"""Seeded synthetic inputs: model shapes, random-init weights, prompts.

This module only *makes inputs*.  It holds none of the decoding method's
arithmetic, so both the HIP path (through the Python binding) and the CPU
oracle may consume what it produces.  Random-init weights stand in for the
fine-tuned CodeLlama checkpoints the paper evaluates (Section 3.4, Table 4),
which are not available; random prompts stand in for its HumanEval and
MultiPL-E infilling prompts.

Weights are i.i.d. N(0, std) (std is the standard deviation), drawn as
float32, scaled, and for bf16 models rounded to bf16 with round-to-nearest-
even.  Every tensor is cut into fixed chunks of ``CHUNK`` elements and chunk
``c`` of tensor ``t`` draws from ``PCG64(SeedSequence([seed, t, c]))``, so the
values do not depend on how many threads generate them.  RMSNorm gains are 1
unless ``gain_std`` > 0, in which case they are ``1 + N(0, gain_std)`` (tests
use this so that a dropped gain cannot go unnoticed).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

CHUNK = 1 << 22
_PROMPT_STREAM = 1_000_003


@dataclass(frozen=True)
class ModelShape:
    """Llama-style decoder shape (no GQA: n_kv_heads == n_heads)."""
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int          # LM-head width V
    n_adaptive: int     # extra embedding rows V..V+A-1 (adaptive token ids)
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    dtype: str = "bf16"  # "fp32" or "bf16": storage type of weights and KV cache


@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    seed: int
    batch: int
    k: int
    prompt_len: int
    max_new: int
    mode: str = "greedy"          # "greedy" or "nucleus"
    temperature: float = 1.0
    top_p: float = 1.0
    top_k: int = 0
    weight_std: float = 0.02
    gain_std: float = 0.0


TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=688,
                  vocab=1024, n_adaptive=5, rms_eps=1e-5, rope_base=10000.0, dtype="fp32")
LLAMA7B = ModelShape(n_layers=32, d_model=4096, n_heads=32, head_dim=128, d_ffn=11008,
                     vocab=32016, n_adaptive=5, rms_eps=1e-5, rope_base=1e6, dtype="bf16")
LLAMA13B = ModelShape(n_layers=40, d_model=5120, n_heads=40, head_dim=128, d_ffn=13824,
                      vocab=32016, n_adaptive=10, rms_eps=1e-5, rope_base=1e6, dtype="bf16")

WORKLOADS = {
    # tiny fp32 decoder, greedy k=5, 64 new tokens
    "tiny": Workload("tiny", TINY, seed=0, batch=1, k=5, prompt_len=32, max_new=64),
    # CodeLlama-7B shape, bf16, greedy k=5, prompt 512, 256 new tokens
    "7b": Workload("7b", LLAMA7B, seed=1, batch=1, k=5, prompt_len=512, max_new=256),
    # CodeLlama-13B shape, bf16, greedy k=10, prompt 2048, 512 new tokens
    "13b": Workload("13b", LLAMA13B, seed=2, batch=1, k=10, prompt_len=2048, max_new=512),
    # 7B shape, batch 4, nucleus top-p 0.95 T 0.8, k=5, prompts 1024, 256 new each
    "7b_bs4_nucleus": Workload("7b_bs4_nucleus", LLAMA7B, seed=3, batch=4, k=5, prompt_len=1024,
                               max_new=256, mode="nucleus", temperature=0.8, top_p=0.95),
    # 7B shape, batch 1, the nucleus settings of the paper's speed comparison (Section 3.4.2, Table 4):
    # top-k 10, top-p 0.95, temperature 0.2 or 1, k=5, prompt 512, 256 new tokens
    "7b_topk10_T0.2": Workload("7b_topk10_T0.2", LLAMA7B, seed=5, batch=1, k=5, prompt_len=512, max_new=256,
                               mode="nucleus", temperature=0.2, top_p=0.95, top_k=10),
    "7b_topk10_T1": Workload("7b_topk10_T1", LLAMA7B, seed=6, batch=1, k=5, prompt_len=512, max_new=256,
                             mode="nucleus", temperature=1.0, top_p=0.95, top_k=10),
}


def tensor_names(shape: ModelShape) -> list[str]:
    """Fixed tensor order: embed, per layer {attn_norm, wq, wk, wv, wo, ffn_norm,
    w_gate, w_up, w_down}, final_norm, lm_head."""
    names = ["embed"]
    for i in range(shape.n_layers):
        names += [f"l{i}.{n}" for n in
                  ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")]
    names += ["final_norm", "lm_head"]
    return names


def tensor_shape(shape: ModelShape, name: str) -> tuple[int, ...]:
    d, f = shape.d_model, shape.d_ffn
    base = name.split(".")[-1]
    return {
        "embed": (shape.vocab + shape.n_adaptive, d),
        "attn_norm": (d,), "ffn_norm": (d,), "final_norm": (d,),
        "wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
        "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
        "lm_head": (shape.vocab, d),
    }[base]


def is_gain(name: str) -> bool:
    return name.split(".")[-1] in ("attn_norm", "ffn_norm", "final_norm")


def _bf16_bits_inplace(x32: np.ndarray, tmp: np.ndarray, out16: np.ndarray) -> None:
    """Round float32 ``x32`` to bf16 (RNE; inputs are finite) and store the bit patterns."""
    u = x32.view(np.uint32)
    np.right_shift(u, 16, out=tmp)
    tmp &= 1
    tmp += 0x7FFF
    tmp += u
    tmp >>= 16
    out16[:] = tmp


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def fill_tensor(wl: Workload, name: str, out: np.ndarray) -> np.ndarray:
    """Fill ``out`` (uint16 bf16 bits for bf16 models, float32 otherwise) with tensor ``name``."""
    shape = wl.shape
    names = tensor_names(shape)
    t_index = names.index(name)
    n = int(np.prod(tensor_shape(shape, name)))
    flat = out.reshape(-1)
    assert flat.size == n
    bf16 = shape.dtype == "bf16"
    assert flat.dtype == (np.uint16 if bf16 else np.float32)
    gain = is_gain(name)
    std = wl.gain_std if gain else wl.weight_std
    n_chunks = (n + CHUNK - 1) // CHUNK

    def work(chunks):
        buf = np.empty(min(CHUNK, n), np.float32)
        tmp = np.empty(min(CHUNK, n), np.uint32) if bf16 else None
        for c in chunks:
            lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
            b = buf[: hi - lo]
            if gain and std == 0.0:
                b[:] = 1.0
            else:
                g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, t_index, c])))
                g.standard_normal(dtype=np.float32, out=b)
                b *= np.float32(std)
                if gain:
                    b += np.float32(1.0)
            if bf16:
                _bf16_bits_inplace(b, tmp[: hi - lo], flat[lo:hi])
            else:
                flat[lo:hi] = b

    nw = min(_workers(), n_chunks)
    if nw <= 1:
        work(range(n_chunks))
    else:
        with ThreadPoolExecutor(nw) as ex:
            list(ex.map(work, [range(i, n_chunks, nw) for i in range(nw)]))
    return out


def tensor(wl: Workload, name: str) -> np.ndarray:
    """Allocate and generate one tensor (uint16 bf16 bits or float32)."""
    dt = np.uint16 if wl.shape.dtype == "bf16" else np.float32
    out = np.empty(tensor_shape(wl.shape, name), dt)
    return fill_tensor(wl, name, out)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 values."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def prompts(wl: Workload, batch: int | None = None, length: int | None = None) -> np.ndarray:
    """Prompt token ids, int32 [batch, length], uniform in [0, V)."""
    b = wl.batch if batch is None else batch
    p = wl.prompt_len if length is None else length
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, _PROMPT_STREAM])))
    return g.integers(0, wl.shape.vocab, size=(b, p), dtype=np.int64).astype(np.int32)


def adaptive_ids(shape: ModelShape, k: int, identical: bool = False) -> np.ndarray:
    """Adaptive token ids a_1..a_k: V..V+k-1 (diverse, needs k <= A) or all V (identical)."""
    if identical:
        return np.full(k, shape.vocab, np.int32)
    assert k <= shape.n_adaptive, "diverse adaptive ids need k <= n_adaptive"
    return (shape.vocab + np.arange(k)).astype(np.int32)


def small_shape(**kw) -> ModelShape:
    """A reduced shape for tests (defaults: the tiny fp32 shape)."""
    return replace(TINY, **kw)


def workload(name: str, **kw) -> Workload:
    return replace(WORKLOADS[name], **kw)


def device_weights(wl: Workload, device="cuda"):
    """Generate every tensor and upload it, in the fixed order, as torch tensors
    (bfloat16 or float32 matrices, float32 gains).  One pinned staging buffer is
    reused for all tensors."""
    import torch
    shape = wl.shape
    names = tensor_names(shape)
    bf16 = shape.dtype == "bf16"
    biggest = max(int(np.prod(tensor_shape(shape, n))) for n in names)
    host_dt = torch.int16 if bf16 else torch.float32
    stage = torch.empty(biggest, dtype=host_dt, pin_memory=torch.cuda.is_available())
    stage_np = stage.numpy().view(np.uint16 if bf16 else np.float32)
    out = []
    for n in names:
        shp = tensor_shape(shape, n)
        cnt = int(np.prod(shp))
        if is_gain(n):
            w = tensor(wl, n)
            host = torch.from_numpy(bf16_bits_to_f32(w) if bf16 else w)
            out.append(host.to(device))
            continue
        fill_tensor(wl, n, stage_np[:cnt])
        dev = torch.empty(shp, dtype=torch.bfloat16 if bf16 else torch.float32, device=device)
        src = stage[:cnt].view(torch.bfloat16) if bf16 else stage[:cnt]
        dev.view(-1).copy_(src, non_blocking=False)
        out.append(dev)
    return out
