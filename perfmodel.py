"""Work accounting for the MoSA layer: algorithmic bytes and FLOPs per kernel
launch (the roofline of every stage), and the paper's FLOP model.

Algorithmic bytes count each input once and each output once (activations,
weights, compact k-sized per-head tensors); they exclude re-reads a kernel
does for its tiling and the T x T / k x d intermediates the method avoids.
FLOPs: 2 per multiply-add; attention counts only the causally allowed
(query, key) pairs.  The paper's own FLOP model (Section 3.2 and Appendix A)
is `paper_flops_*` below.
"""
from dataclasses import dataclass

HBM_PEAK = 8.0e12  # bytes/s, MI355X HBM3E
MFMA_PEAK = {"bf16": 2.5e15, "f32": 157.3e12}  # dense FLOP/s by operand type


@dataclass
class StageWork:
    name: str
    bytes: float
    flops: float


def _pairs(n, causal):
    return n * (n + 1) / 2 if causal else n * n


def stage_work(w, with_backward=True):
    """Algorithmic work of every kernel the library times, keyed by stage name.
    The output side (out_proj + out_combine) and the dX side (dx_proj +
    dx_combine) are accounted as one stage each (GROUPS): their algorithmic
    bytes are those of the paper's operation (A, W^O and Y once; the per-head
    k x d rows that the two-kernel design writes and reads back are not
    algorithmic traffic)."""
    es = 2 if w.dtype == "bf16" else 4
    B, T, d, H, dh, k, Hd = w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.dense_heads
    X = B * T * d * es
    rows = B * H * k  # selected rows over all heads
    out = {}

    def add(name, nbytes, flops):
        out[name] = StageWork(name, float(nbytes), float(flops))

    if H:
        add("router", X + H * d * es + B * H * T * 4 + B * T * 4, 2.0 * B * T * H * d)
        add("select", B * H * T * 4 + B * T * 4 + H * d * es + rows * 8 + B * H * T * 2, 0.0)
        add("qkv", X + 3 * H * d * dh * es + 3 * rows * dh * es + rows * 4, 2.0 * rows * d * 3 * dh)
        add("attn", 4 * rows * dh * es + rows * 4, 4.0 * dh * _pairs(k, w.causal) * B * H)
    if Hd:
        add("qkv_dense", X + 3 * Hd * d * dh * es + 3 * B * Hd * T * dh * es, 2.0 * B * Hd * T * d * 3 * dh)
        add("attn_dense", 4 * B * Hd * T * dh * es + B * Hd * T * 4, 4.0 * dh * _pairs(T, w.causal) * B * Hd)
    add("out_scatter",
        rows * dh * es + rows * 8 + H * dh * d * es + B * Hd * T * dh * es + Hd * dh * d * es + X,
        2.0 * rows * dh * d + 2.0 * B * Hd * T * dh * d)
    if not with_backward:
        return out
    if H:
        add("bwd_out", X + H * dh * d * es + 2 * rows * dh * es + rows * 16, 2.0 * rows * d * dh)
        add("attn_bwd_kv", 6 * rows * dh * es + rows * 8, 8.0 * dh * _pairs(k, w.causal) * B * H)
        add("attn_bwd_q", 5 * rows * dh * es + rows * 8, 6.0 * dh * _pairs(k, w.causal) * B * H)
        add("wgrad_qkv", X + 3 * rows * dh * es + rows * 4 + 3 * H * d * dh * es + H * d * es,
            2.0 * rows * d * (3 * dh + 1))
        add("wgrad_o", X + rows * dh * es + rows * 4 + H * dh * d * es, 2.0 * rows * dh * d)
    if Hd:
        R = B * Hd * T
        add("bwd_out_dense", X + Hd * dh * d * es + 2 * R * dh * es + R * 4, 2.0 * R * d * dh)
        add("attn_bwd_kv_dense", 6 * R * dh * es + R * 8, 8.0 * dh * _pairs(T, w.causal) * B * Hd)
        add("attn_bwd_q_dense", 5 * R * dh * es + R * 8, 6.0 * dh * _pairs(T, w.causal) * B * Hd)
        add("wgrad_qkv_dense", X + 3 * R * dh * es + 3 * Hd * d * dh * es, 2.0 * R * d * 3 * dh)
        add("wgrad_o_dense", X + R * dh * es + Hd * dh * d * es, 2.0 * R * dh * d)
    add("dx_scatter",
        3 * rows * dh * es + rows * 8 + 3 * H * d * dh * es + H * d * es
        + 3 * B * Hd * T * dh * es + 3 * Hd * d * dh * es + X,
        2.0 * rows * 3 * dh * d + 2.0 * rows * d + 2.0 * B * Hd * T * 3 * dh * d)
    return out


# Stages made of two kernels (the library records one event per kernel).
GROUPS = {"out_scatter": ("out_proj", "out_combine"), "dx_scatter": ("dx_proj", "dx_combine")}


def group_stage_times(kernel_ms):
    """Per-stage times from per-kernel times: a group is the sum of its kernels."""
    out = {}
    for name, ms in kernel_ms.items():
        for g, members in GROUPS.items():
            if name in members:
                out[g] = out.get(g, 0.0) + ms
                break
        else:
            out[name] = ms
    return out


def roofline(stage: StageWork, seconds: float, dtype: str):
    """Binding roofline of one stage at a measured time."""
    peak_f = MFMA_PEAK[dtype]
    ridge = peak_f / HBM_PEAK
    ai = stage.flops / stage.bytes if stage.bytes else float("inf")
    if stage.flops > 0 and ai >= ridge:
        achieved = stage.flops / seconds
        return {"bound": "mfma", "achieved": achieved / 1e12, "peak": peak_f / 1e12, "unit": "TFLOP/s",
                "frac": achieved / peak_f, "ai": ai}
    achieved = stage.bytes / seconds
    return {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": achieved / HBM_PEAK, "ai": ai}


# ---------------------------------------------------------------------------
# The paper's FLOP model (Section 3.2 "FLOPs Calculation", Appendix A)
# ---------------------------------------------------------------------------

def paper_flops_dense_head(h, hp, T):
    """Q, K, V, O mappings 8 h h' T plus attention 4 h' T^2."""
    return 8 * h * hp * T + 4 * hp * T * T


def paper_flops_mosa_head(h, hp, T, k):
    """Mappings 8 h h' k, attention 4 h' k^2, routing overhead 2 h T + h' k."""
    return 8 * h * hp * k + 4 * hp * k * k + 2 * h * T + hp * k


def paper_flops_model(layers, h, hp, T, dense_heads, mosa_heads=0, k=0):
    """Forward FLOPs of a whole model: attention heads per layer plus the
    4h feed-forward block 16 h^2 T (Appendix A)."""
    return (layers * dense_heads * paper_flops_dense_head(h, hp, T)
            + layers * mosa_heads * (paper_flops_mosa_head(h, hp, T, k) if mosa_heads else 0)
            + 16 * layers * h * h * T)


def paper_mosa_heads_for_budget(layers, h, hp, T, baseline_heads, dense_heads, sparsity):
    """Largest number of MoSA heads whose model does not exceed the FLOPs of the
    dense baseline with `baseline_heads` heads (Section 3.2, Appendix A)."""
    budget = paper_flops_model(layers, h, hp, T, baseline_heads)
    k = T // sparsity
    fixed = paper_flops_model(layers, h, hp, T, dense_heads)
    return int((budget - fixed) // (layers * paper_flops_mosa_head(h, hp, T, k)))
