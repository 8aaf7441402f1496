"""Seeded synthetic inputs for the GoCkpt hot path (tests, smoke check, bench).

Holds none of the method's arithmetic: it only draws numbers and lays out
tensors.  Both the HIP path and the oracle receive the same arrays from here.

The paper trains LLaMA3.x-1B, Qwen3-0.6B, OPT-350M and LLaMA3-8B on Wikidata
(Sec. 5.2); neither the data nor the weights are available, and the method
never looks at values beyond their layout, so model-shaped synthetic
parameter sets stand in for them:

  * ``flat16m``   one fp32 vector of 16,777,216 elements;
  * ``gpt1p3b``   GPT-style 1.3B: vocab 50304, hidden 2048, ffn 8192, 24 layers
                   (qkv, proj, fc1, fc2 matrices; two LayerNorms with bias);
  * ``llama7b``   Llama-style 7B: vocab 32000, hidden 4096, ffn 11008, 32 layers
                   (q, k, v, o; gate, up, down; two RMSNorms), untied head;
  * ``llama13b``  as llama7b with hidden 5120, ffn 13824, 40 layers.

Values: master ~ N(0, 0.02); gradients bf16 (or fp16) ~ N(0, 1e-3) (times
the loss scale when dynamic scaling is on) or Laplace(0, 5e-4); +inf planted
at a seeded index on chosen steps.  Host draws use numpy's Philox and
torch's float32 -> bfloat16 conversion (numpy's for float16); device draws
of full-size gradients use a Philox4x32-10 kernel of the bench helper library
with HIP's own conversions.  The two are different draws of the same laws;
a test always hands the same arrays to both sides.
"""
from __future__ import annotations

import numpy as np

# ---- layouts -------------------------------------------------------------------


def layout_flat(n: int = 16_777_216):
    return [("params", int(n))]


def layout_gpt(layers: int = 24, hidden: int = 2048, ffn: int = 8192, vocab: int = 50304):
    h = hidden
    out = [("wte", vocab * h)]
    for i in range(layers):
        p = f"h{i}."
        out += [(p + "ln1.w", h), (p + "ln1.b", h), (p + "qkv", 3 * h * h), (p + "proj", h * h),
                (p + "ln2.w", h), (p + "ln2.b", h), (p + "fc1", ffn * h), (p + "fc2", h * ffn)]
    out += [("ln_f.w", h), ("ln_f.b", h)]
    return out


def layout_llama(layers: int = 32, hidden: int = 4096, ffn: int = 11008, vocab: int = 32000):
    h = hidden
    out = [("embed", vocab * h)]
    for i in range(layers):
        p = f"l{i}."
        out += [(p + "attn_norm", h), (p + "q", h * h), (p + "k", h * h), (p + "v", h * h), (p + "o", h * h),
                (p + "ffn_norm", h), (p + "gate", ffn * h), (p + "up", ffn * h), (p + "down", h * ffn)]
    out += [("norm", h), ("lm_head", vocab * h)]
    return out


LAYOUTS = {
    "flat16m": layout_flat,
    "gpt1p3b": layout_gpt,
    "llama7b": layout_llama,
    "llama13b": lambda: layout_llama(40, 5120, 13824, 32000),
}


def tensor_ends(layout) -> np.ndarray:
    return np.cumsum([n for _, n in layout], dtype=np.int64)


def numel(layout) -> int:
    return int(sum(n for _, n in layout))


# ---- workload configurations ------------------------------------------------------

WORKLOADS = {
    # name: layout, K, partition, gradient law, dynamic scaling, inf steps, ring
    "flat16m_k4": dict(layout="flat16m", K=4, partition="equal", grad="normal", dynamic=False,
                       inf_steps=(), ring_bytes=256 << 20),
    "gpt1p3b_k8": dict(layout="gpt1p3b", K=8, partition="bytes", grad="normal", dynamic=False,
                       inf_steps=(), ring_bytes=24 << 30),
    "llama7b_k16": dict(layout="llama7b", K=16, partition="bytes", grad="normal", dynamic=False,
                        inf_steps=(), ring_bytes=256 << 20),
    "gpt1p3b_k8_dynscale": dict(layout="gpt1p3b", K=8, partition="bytes", grad="normal", dynamic=True,
                                inf_steps=(3, 7), ring_bytes=24 << 30),
    "llama13b_k32": dict(layout="llama13b", K=32, partition="tensors", grad="laplace", dynamic=False,
                         inf_steps=(), ring_bytes=None),
}

# Loss scale the c4-style gradients carry at window step s: initial 65536,
# halved after each planted inf (steps 3 and 7 are skipped), growth interval
# 1000 never reached inside the window.
DYNSCALE_SCHEDULE = {1: 65536.0, 2: 65536.0, 3: 65536.0, 4: 32768.0, 5: 32768.0, 6: 32768.0, 7: 32768.0,
                     8: 16384.0}


def _seed(*parts: int) -> int:
    s = 0x9E3779B97F4A7C15
    for p in parts:
        s = (s * 6364136223846793005 + (int(p) & 0xFFFFFFFFFFFFFFFF) + 1442695040888963407) % (1 << 64)
    return s >> 1


def _rng(*parts: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=_seed(*parts)))


def _bf16_bits_cpu(x: np.ndarray) -> np.ndarray:
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16) \
        .numpy().view(np.uint16)


# ---- host generators (sizes the oracle handles) ------------------------------------


def master_cpu(n: int, seed: int = 0, std: float = 0.02) -> np.ndarray:
    return (_rng(seed, 0).standard_normal(n, dtype=np.float32) * np.float32(std)).astype(np.float32)


def inf_index(n: int, seed: int, step: int) -> int:
    return int(_rng(seed, 2, step).integers(0, n))


def grads_cpu(n: int, seed: int, step: int, law: str = "normal", scale: float = 1.0,
              plant_inf: bool = False, sigma: float = 1e-3, laplace_b: float = 5e-4,
              dtype: str = "bf16") -> np.ndarray:
    """16-bit patterns (bf16, or fp16 with dtype="fp16") of one step's gradients."""
    r = _rng(seed, 1, step)
    if law == "normal":
        x = r.standard_normal(n, dtype=np.float32) * np.float32(sigma)
    elif law == "laplace":
        x = r.laplace(0.0, laplace_b, n).astype(np.float32)
    else:
        raise ValueError(law)
    x = (x * np.float32(scale)).astype(np.float32)
    if dtype == "fp16":
        # a loss scale grown too large overflows to inf here, as a scaled
        # fp16 backward does: the step is then skipped
        with np.errstate(over="ignore"):
            g = x.astype(np.float16).view(np.uint16)
    elif dtype == "bf16":
        g = _bf16_bits_cpu(x)
    else:
        raise ValueError(dtype)
    if plant_inf:
        g[inf_index(n, seed, step)] = 0x7C00 if dtype == "fp16" else 0x7F80
    return g


# ---- device generators (full sizes; torch's device RNG, in slices) --------------------

_SLICE = 1 << 28


def master_dev_(out, seed: int = 0, std: float = 0.02) -> None:
    """Fill a float32 device tensor with N(0, std) on the current stream."""
    import torch
    g = torch.Generator(device=out.device)
    g.manual_seed(_seed(seed, 0) & 0x7FFFFFFFFFFFFFFF)
    n = out.numel()
    for a in range(0, n, _SLICE):
        b = min(n, a + _SLICE)
        torch.randn(b - a, generator=g, device=out.device, dtype=torch.float32, out=out[a:b])
        out[a:b].mul_(std)


_BENCH_LIB = None


def _bench_lib():
    """The harness's device helpers (libgockpt_bench.so): the gradient
    generator kernel."""
    global _BENCH_LIB
    if _BENCH_LIB is None:
        import ctypes
        import os
        path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2511_07035_amd",
                            "libgockpt_bench.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} missing: python -m paper_2511_07035_amd.build")
        L = ctypes.CDLL(path)
        L.gockpt_bench_fill_grads.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int,
                                              ctypes.c_float, ctypes.c_float, ctypes.c_int, ctypes.c_int64,
                                              ctypes.c_void_p]
        L.gockpt_bench_fill_grads.restype = ctypes.c_int
        _BENCH_LIB = L
    return _BENCH_LIB


def grads_dev_(out, seed: int, step: int, law: str = "normal", scale: float = 1.0, plant_inf: bool = False,
               sigma: float = 1e-3, laplace_b: float = 5e-4) -> None:
    """Fill a bfloat16 or float16 device tensor (16-byte aligned) with one
    step's gradients on the current stream: N(0, sigma) or Laplace(0,
    laplace_b), times `scale`, drawn by a counter-based generator keyed by
    (seed, step) in one kernel (libgockpt_bench.so), so that generating a
    step's gradients costs about what a backward's writes of them would."""
    import torch
    if out.dtype not in (torch.bfloat16, torch.float16) or not out.is_contiguous():
        raise ValueError("out must be a contiguous bfloat16 or float16 tensor")
    if law not in ("normal", "laplace"):
        raise ValueError(law)
    n = out.numel()
    plant = inf_index(n, seed, step) if plant_inf else -1
    rc = _bench_lib().gockpt_bench_fill_grads(
        out.data_ptr(), n, _seed(seed, 1, step), 0 if law == "normal" else 1,
        sigma if law == "normal" else laplace_b, float(scale), 1 if out.dtype == torch.float16 else 0, plant,
        torch.cuda.current_stream(out.device).cuda_stream)
    if rc != 0:
        raise RuntimeError(f"gockpt_bench_fill_grads failed ({rc})")
