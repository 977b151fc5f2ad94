"""Seeded synthetic workloads for the MoSA layer (shared by tests, smoke and bench).

This module only draws random inputs and describes shapes: it holds none of the
layer's arithmetic.  Values follow the recipe stated for the language-model
workloads of the paper (Section 3, "Implementation details"; Appendix C,
Table 4): activations X ~ N(0, 1) (stand-in for pre-LayerNorm'd activations of
C4 text, which is not available), every weight ~ N(0, 1/d_model), upstream
gradient dY ~ N(0, 1).  Draw order: X, W_r, W_q, W_k, W_v, W_o, then the dense
heads' W_q, W_k, W_v, W_o, then dY -- from one numpy PCG64 generator seeded
with the config's seed.  bf16 tensors are the float32 draws rounded to nearest
even and are carried as uint16 bit patterns, so both sides of every check see
the same stored bits.
"""
from dataclasses import dataclass, asdict

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    seq_len: int
    d_model: int
    heads: int          # MoSA heads
    d_head: int
    k: int              # tokens per MoSA head
    dense_heads: int = 0
    causal: bool = True
    dtype: str = "bf16"  # storage type: "bf16" or "f32"
    backward: bool = False
    seed: int = 0
    # variants of the layer (all off by default): forced first token
    # (Section 3.2), fixed sparse stride (Section 3.1), rotary encoding at the
    # original positions (Section 2.2), local window of the dense heads (Section 3.4)
    first_token: bool = False
    fixed_stride: int = 0
    rope: bool = False
    rope_base: float = 10000.0
    window: int = 0

    def as_dict(self):
        return asdict(self)

    def variants(self):
        return dict(first_token=self.first_token, fixed_stride=self.fixed_stride, rope=self.rope,
                    rope_base=self.rope_base, window=self.window)

    @property
    def tokens(self):
        return self.batch * self.seq_len


# The five workloads: a tiny fp32 check, then bf16 workloads shaped like the
# paper's models (T = 1024, d_head = 64, sparsities 8/16/64 and a long sequence).
WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", 1, 256, 128, 4, 32, 32, dtype="f32", seed=0),
    "fwd_d512": Workload("fwd_d512", 8, 1024, 512, 32, 64, 128, seed=1),
    "fwdbwd_d1024": Workload("fwdbwd_d1024", 4, 1024, 1024, 128, 64, 64, backward=True, seed=2),
    "hybrid_d1024": Workload("hybrid_d1024", 8, 1024, 1024, 256, 64, 16, dense_heads=4,
                             backward=True, seed=3),
    "long_t8192": Workload("long_t8192", 1, 8192, 1024, 64, 64, 512, seed=4),
    # the fwd_d512 shape in the paper's IsoFLOP setting (rotary encoding at the
    # original positions, token 0 always kept), and as fixed sparse attention
    # with stride 8 (I = 0, 8, ..., 1016; r = 1)
    "fwd_d512_rope_first": Workload("fwd_d512_rope_first", 8, 1024, 512, 32, 64, 128, seed=1,
                                    first_token=True, rope=True),
    "fixed_d512": Workload("fixed_d512", 8, 1024, 512, 32, 64, 128, seed=1, fixed_stride=8),
    # the long-sequence hybrid of Section 3.4: 60 MoSA heads with k = 64 beside
    # 4 local (sliding-window) heads, d_model 1024, T = 8192 (window 512: the
    # paper does not state it)
    "long_local_t8192": Workload("long_local_t8192", 1, 8192, 1024, 60, 64, 64, dense_heads=4,
                                 backward=True, seed=4, window=512),
    # the dense causal layer that the long-sequence MoSA layer is compared
    # with: by the paper's FLOP formula (Appendix A) 64 MoSA heads with
    # k = 512 cost about as much as one dense head at T = 8192
    "long_dense1_t8192": Workload("long_dense1_t8192", 1, 8192, 1024, 0, 64, 0, dense_heads=1, seed=4),
}

# Workloads timed together with a comparator on the same GPU (equal FLOPs by
# the paper's formula, Appendix A).
COMPARATORS = {"long_t8192": "long_dense1_t8192"}


def f32_to_bf16_bits(a):
    """Round float32 values to the nearest bf16 (ties to even); return uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits):
    """Exact widening of bf16 bit patterns to float32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def as_f32(a):
    """Exact float32 view of a stored tensor (float32 or bf16 bits)."""
    return bf16_bits_to_f32(a) if a.dtype == np.uint16 else np.asarray(a, dtype=np.float32)


def _store(x, dtype):
    return f32_to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_inputs(w: Workload, seed=None, with_grad=None):
    """Draw the inputs of workload ``w``.  Returns a dict of numpy arrays:
    X [B,T,d]; Wr [H,d]; Wq/Wk/Wv [H,d,dh]; Wo [H,dh,d]; Wq_d/Wk_d/Wv_d [Hd,d,dh],
    Wo_d [Hd,dh,d] (None when there are no dense heads); dY [B,T,d] when
    ``with_grad`` (default: w.backward)."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    B, T, d, H, dh, Hd = w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.dense_heads
    wstd = 1.0 / np.sqrt(d)

    def normal(shape, std=1.0):
        return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)

    out = {"X": _store(normal((B, T, d)), w.dtype)}
    out["Wr"] = _store(normal((H, d), wstd), w.dtype)
    out["Wq"] = _store(normal((H, d, dh), wstd), w.dtype)
    out["Wk"] = _store(normal((H, d, dh), wstd), w.dtype)
    out["Wv"] = _store(normal((H, d, dh), wstd), w.dtype)
    out["Wo"] = _store(normal((H, dh, d), wstd), w.dtype)
    if Hd > 0:
        out["Wq_d"] = _store(normal((Hd, d, dh), wstd), w.dtype)
        out["Wk_d"] = _store(normal((Hd, d, dh), wstd), w.dtype)
        out["Wv_d"] = _store(normal((Hd, d, dh), wstd), w.dtype)
        out["Wo_d"] = _store(normal((Hd, dh, d), wstd), w.dtype)
    else:
        out["Wq_d"] = out["Wk_d"] = out["Wv_d"] = out["Wo_d"] = None
    if w.backward if with_grad is None else with_grad:
        out["dY"] = _store(normal((B, T, d)), w.dtype)
    return out


def small(name="small", batch=2, seq_len=96, d_model=64, heads=3, d_head=32, k=20,
          dense_heads=0, causal=True, dtype="bf16", backward=True, seed=11, **variants):
    """A small workload for fast checks (``variants``: the Workload variant fields)."""
    return Workload(name, batch, seq_len, d_model, heads, d_head, k, dense_heads, causal, dtype,
                    backward, seed, **variants)
