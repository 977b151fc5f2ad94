// C ABI of the MoSA layer: argument validation, workspace carve-up and the
// launch sequence of the forward and backward passes (see include/mosa.h).
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "kernels.h"
#include "mosa.h"

namespace {

using namespace mosa;

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
    mosa_saved_layout saved;
    // forward scratch
    size_t z, xnorm, unc_tok, unc_key, unc_sel, Xo, ybase, apart, apart_d;
    // backward scratch
    size_t dA, D, dz, dz16, dQKV, dXs, dAd, Dd, dQKVd, wpart, wpart_d, dxbase, dwr;
    size_t fwd_scratch, scratch_total;
};

class Carver {
  public:
    size_t take(size_t bytes) {
        size_t at = off_;
        off_ = align_up(off_ + bytes);
        return at;
    }
    size_t total() const { return off_; }

  private:
    size_t off_ = 0;
};

int validate_shape(const mosa_shape* s) {
    if (!s) return MOSA_ERR_INVALID_ARG;
    if (s->dtype != MOSA_F32 && s->dtype != MOSA_BF16) return MOSA_ERR_INVALID_ARG;
    if (s->batch < 1 || s->seq_len < 1 || s->d_model < 1 || s->d_head < 1) return MOSA_ERR_INVALID_ARG;
    if (s->heads < 0 || s->dense_heads < 0 || s->heads + s->dense_heads < 1) return MOSA_ERR_INVALID_ARG;
    if (s->causal != 0 && s->causal != 1) return MOSA_ERR_INVALID_ARG;
    if (s->heads > 0 && (s->k < 1 || s->k > s->seq_len)) return MOSA_ERR_INVALID_ARG;
    if (s->d_head != 32 && s->d_head != 64) return MOSA_ERR_UNSUPPORTED;
    if (s->d_model % 64 != 0) return MOSA_ERR_UNSUPPORTED;
    if (s->seq_len > 16384) return MOSA_ERR_UNSUPPORTED;
    // index arithmetic inside the kernels uses 32-bit row counts
    const double rows = (double)s->batch * s->seq_len * (double)(s->heads > s->dense_heads ? s->heads : s->dense_heads);
    if (rows > 2.0e9) return MOSA_ERR_UNSUPPORTED;
    // row counts of one head (B * k or B * T) are divided with a float reciprocal
    if ((double)s->batch * s->seq_len >= 16777216.0) return MOSA_ERR_UNSUPPORTED;
    // variants
    if (s->first_token != 0 && s->first_token != 1) return MOSA_ERR_INVALID_ARG;
    if (s->rope != 0 && s->rope != 1) return MOSA_ERR_INVALID_ARG;
    if (s->fixed_stride < 0 || s->window < 0) return MOSA_ERR_INVALID_ARG;
    if (s->rope && !(s->rope_base > 1.0f)) return MOSA_ERR_INVALID_ARG;
    if (s->window > 0 && !s->causal) return MOSA_ERR_INVALID_ARG;
    if (s->heads > 0 && s->fixed_stride > 0 &&
        (s->first_token || (long long)(s->k - 1) * s->fixed_stride > s->seq_len - 1))
        return MOSA_ERR_INVALID_ARG;
    return MOSA_OK;
}

bool routed(const mosa_shape* s) { return s->heads > 0 && s->fixed_stride == 0; }

Layout make_layout(const mosa_shape* s) {
    const size_t B = s->batch, T = s->seq_len, d = s->d_model, H = s->heads, Hd = s->dense_heads, dh = s->d_head;
    const size_t k = s->heads > 0 ? (size_t)s->k : 0;
    const size_t es = s->dtype == MOSA_BF16 ? 2 : 4;
    Layout L;
    Carver sv;
    L.saved.I = sv.take(B * H * k * 4);
    L.saved.r = sv.take(B * H * k * 4);
    L.saved.slot = sv.take(B * H * T * 2);
    L.saved.QKV = sv.take(B * H * k * 3 * dh * es);
    L.saved.A = sv.take(B * H * k * dh * es);
    L.saved.lse = sv.take(B * H * k * 4);
    L.saved.QKVd = sv.take(B * Hd * T * 3 * dh * es);
    L.saved.Ad = sv.take(B * Hd * T * dh * es);
    L.saved.lsed = sv.take(B * Hd * T * 4);
    L.saved.rope = sv.take(s->rope ? T * (dh / 4) * 8 : 0);  // (cos, sin) table
    L.saved.status = sv.take(B * H * 4);                      // selection status per (b, h)
    L.saved.total = sv.total();

    // forward and backward scratch share the same buffer (used at different times)
    Carver fw;
    L.z = fw.take(B * H * T * 4);
    L.xnorm = fw.take(B * T * 4);
    L.unc_tok = fw.take(B * H * T * 4);
    L.unc_key = fw.take(B * H * T * 8);
    L.unc_sel = fw.take(B * H * T * 4);
    L.Xo = fw.take(B * H * k * d * es);
    L.ybase = fw.take(Hd > 0 ? B * T * d * es : 0);  // dense heads' part of Y
    {  // partial results of the attention's key splits, MoSA and dense heads
       // apart (the two chains may run at the same time)
        const int dt = s->dtype == MOSA_BF16 ? kBF16 : kF32;
        L.apart = fw.take(H > 0 ? attn_fwd_part_bytes(dt, (int)(B * H), (int)k, (int)dh, s->causal, 0) : 0);
        L.apart_d = fw.take(Hd > 0 ? attn_fwd_part_bytes(dt, (int)(B * Hd), (int)T, (int)dh, s->causal, s->window) : 0);
    }
    Carver bw;
    L.dA = bw.take(B * H * k * dh * es);
    L.D = bw.take(B * H * k * 4);
    L.dz = bw.take(B * H * k * 4);
    L.dz16 = bw.take(B * H * k * 16 * es);
    L.dQKV = bw.take(B * H * k * 3 * dh * es);
    L.dXs = bw.take(B * H * k * d * es);
    L.dAd = bw.take(B * Hd * T * dh * es);
    L.Dd = bw.take(B * Hd * T * 4);
    L.dQKVd = bw.take(B * Hd * T * 3 * dh * es);
    L.dxbase = bw.take(Hd > 0 ? B * T * d * es : 0);  // dense heads' part of dX
    L.dwr = bw.take(H > 0 && s->fixed_stride > 0 ? H * d * es : 0);  // dW^r sink without a router
    {
        const int dt = s->dtype == MOSA_BF16 ? kBF16 : kF32;
        L.wpart = bw.take(wgrad_partial_bytes(dt, (int)B, (int)d, (int)H, (int)dh, (int)k, 1));
        L.wpart_d = bw.take(wgrad_partial_bytes(dt, (int)B, (int)d, (int)Hd, (int)dh, (int)T, 0));
    }
    L.fwd_scratch = fw.total();
    L.scratch_total = fw.total() > bw.total() ? fw.total() : bw.total();
    return L;
}

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int check_weights(const mosa_shape* s, const mosa_weights* w) {
    if (!w) return MOSA_ERR_INVALID_ARG;
    if (s->heads > 0) {
        const void* need[4] = {w->Wq, w->Wk, w->Wv, w->Wo};
        for (const void* p : need)
            if (!p || !aligned(p, 16)) return MOSA_ERR_INVALID_ARG;
        // fixed sparse attention has no router: W^r may be NULL
        if ((routed(s) && !w->Wr) || (w->Wr && !aligned(w->Wr, 16))) return MOSA_ERR_INVALID_ARG;
    }
    if (s->dense_heads > 0) {
        const void* need[4] = {w->Wq_d, w->Wk_d, w->Wv_d, w->Wo_d};
        for (const void* p : need)
            if (!p || !aligned(p, 16)) return MOSA_ERR_INVALID_ARG;
    }
    return MOSA_OK;
}

template <typename T>
T* at(void* base, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}
template <typename T>
const T* at(const void* base, size_t off) {
    return reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}

// Records a caller-created hipEvent_t after every kernel launch (timed
// variants only); a call without events records nothing.
struct StageMarks {
    mosa_stage_events* ev;
    hipStream_t stream;
    int mark(const char* name) {
        if (!ev) return 0;
        if (ev->count >= MOSA_MAX_STAGES || !ev->events[ev->count]) return 1;
        ev->names[ev->count] = name;
        return hipEventRecord(static_cast<hipEvent_t>(ev->events[ev->count++]), stream) != hipSuccess;
    }
    static int hook(void* ctx, const char* name) { return static_cast<StageMarks*>(ctx)->mark(name); }
    Marker marker() { return Marker{&StageMarks::hook, this}; }
};

// The dense heads' chain of kernels is independent of the MoSA heads' until
// the head-ordered sum, so the untimed calls run it on an auxiliary stream of
// the device (fork and join through two events), and the two chains share the
// CUs.  Per device, created at the first call that has both kinds of heads and
// kept until the process ends; the enqueue of a call is serialised under the
// mutex, so that one call's fork and join events are not re-recorded by
// another host thread in between.  Default priority, like every stream here.
struct AuxStream {
    hipStream_t s = nullptr;
    hipEvent_t fork = nullptr, join = nullptr, mid = nullptr;  // mid: a point inside the auxiliary chain
    bool tried = false, ok = false;
};
constexpr int kMaxDevices = 64;
std::mutex g_aux_mu;
AuxStream g_aux[kMaxDevices];

// The current device's auxiliary stream (g_aux_mu held), or nullptr.
AuxStream* aux_stream() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    AuxStream& a = g_aux[dev];
    if (!a.tried) {
        a.tried = true;
        a.ok = hipStreamCreateWithFlags(&a.s, hipStreamNonBlocking) == hipSuccess &&
               hipEventCreateWithFlags(&a.fork, hipEventDisableTiming) == hipSuccess &&
               hipEventCreateWithFlags(&a.join, hipEventDisableTiming) == hipSuccess &&
               hipEventCreateWithFlags(&a.mid, hipEventDisableTiming) == hipSuccess;
    }
    return a.ok ? &a : nullptr;
}

// Fork: work on the returned stream starts after everything enqueued on
// `main` so far.  Join: `main` waits for everything enqueued on `aux`.
int aux_fork(AuxStream* ax, hipStream_t main) {
    return hipEventRecord(ax->fork, main) != hipSuccess || hipStreamWaitEvent(ax->s, ax->fork, 0) != hipSuccess;
}
int aux_join(AuxStream* ax, hipStream_t main) {
    return hipEventRecord(ax->join, ax->s) != hipSuccess || hipStreamWaitEvent(main, ax->join, 0) != hipSuccess;
}

}  // namespace

extern "C" {

const char* mosa_status_string(int status) {
    switch (status) {
        case MOSA_OK: return "ok";
        case MOSA_ERR_INVALID_ARG: return "invalid argument (size, null pointer or alignment)";
        case MOSA_ERR_UNSUPPORTED: return "unsupported shape (d_head must be 32 or 64, d_model a multiple of 64, seq_len <= 16384)";
        case MOSA_ERR_WORKSPACE: return "saved or scratch buffer smaller than mosa_workspace_size";
        case MOSA_ERR_HIP: return "HIP launch failure";
        default: return "unknown status";
    }
}

int mosa_workspace_size(const mosa_shape* s, size_t* saved_bytes, size_t* scratch_bytes) {
    int st = validate_shape(s);
    if (st) return st;
    if (!saved_bytes || !scratch_bytes) return MOSA_ERR_INVALID_ARG;
    Layout L = make_layout(s);
    *saved_bytes = L.saved.total;
    *scratch_bytes = L.scratch_total;
    return MOSA_OK;
}

int mosa_saved_offsets(const mosa_shape* s, mosa_saved_layout* out) {
    int st = validate_shape(s);
    if (st) return st;
    if (!out) return MOSA_ERR_INVALID_ARG;
    *out = make_layout(s).saved;
    return MOSA_OK;
}

}  // extern "C"

namespace mosa {

size_t forward_scratch_bytes(const mosa_shape* s) { return validate_shape(s) ? 0 : make_layout(s).fwd_scratch; }

// The forward (timed when ev != nullptr).  fwd_scratch_only: scratch need only
// hold the forward's part (the allocation-free entry point's static buffer).
int forward_impl(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y, int accumulate,
                 int32_t* I_out, float* r_out, void* saved, size_t saved_bytes, void* scratch,
                 size_t scratch_bytes, void* stream_, mosa_stage_events* ev, bool fwd_scratch_only) {
    int st = validate_shape(s);
    if (st) return st;
    if ((st = check_weights(s, w))) return st;
    if (!X || !Y || !aligned(X, 16) || !aligned(Y, 16)) return MOSA_ERR_INVALID_ARG;
    if (!saved || !scratch || !aligned(saved, kAlign) || !aligned(scratch, kAlign)) return MOSA_ERR_INVALID_ARG;
    if ((I_out && !aligned(I_out, 4)) || (r_out && !aligned(r_out, 4))) return MOSA_ERR_INVALID_ARG;
    const Layout L = make_layout(s);
    if (saved_bytes < L.saved.total || scratch_bytes < (fwd_scratch_only ? L.fwd_scratch : L.scratch_total))
        return MOSA_ERR_WORKSPACE;

    hipStream_t stream = static_cast<hipStream_t>(stream_);
    if (ev) ev->count = 0;
    StageMarks sm{ev, stream};
    int e = sm.mark("start");
    const int B = s->batch, T = s->seq_len, d = s->d_model, H = s->heads, Hd = s->dense_heads, dh = s->d_head;
    const int k = H > 0 ? s->k : 0, dt = s->dtype, causal = s->causal;
    int32_t* I = at<int32_t>(saved, L.saved.I);
    float* r = at<float>(saved, L.saved.r);
    int16_t* slot = at<int16_t>(saved, L.saved.slot);
    void* QKV = at<char>(saved, L.saved.QKV);
    void* A = at<char>(saved, L.saved.A);
    float* lse = at<float>(saved, L.saved.lse);
    void* QKVd = at<char>(saved, L.saved.QKVd);
    void* Ad = at<char>(saved, L.saved.Ad);
    float* lsed = at<float>(saved, L.saved.lsed);
    int32_t* status = at<int32_t>(saved, L.saved.status);
    void* Xo = at<char>(scratch, L.Xo);
    float* apart = at<float>(scratch, L.apart);

    float2* rope = s->rope ? at<float2>(saved, L.saved.rope) : nullptr;
    if (rope) {
        e |= launch_rope_table(T, dh, s->rope_base, rope, stream);
        e |= sm.mark("rope_table");
    }
    // the dense heads on the auxiliary stream (untimed calls with both kinds of heads)
    std::unique_lock<std::mutex> lock(g_aux_mu, std::defer_lock);
    AuxStream* ax = nullptr;
    if (!ev && H > 0 && Hd > 0 && combine_split_ok(d, H)) {
        lock.lock();
        ax = aux_stream();
        if (ax && aux_fork(ax, stream)) return MOSA_ERR_HIP;
    }
    if (Hd > 0) {
        hipStream_t ds = ax ? ax->s : stream;
        // 64-row tiles (twice the workgroups) unless the heads are local:
        // measured faster on 4 causal heads of B = 8, T = 1024 beside the MoSA
        // heads (0.396 -> 0.392 ms cold per step) and on one head of T = 8192
        // alone (0.080 -> 0.074 ms), slower on 4 local heads of T = 8192 beside
        // 60 MoSA heads (0.262 -> 0.268 ms)
        e |= launch_qkv(dt, X, nullptr, w->Wq_d, w->Wk_d, w->Wv_d, B, T, d, Hd, dh, T, QKVd, rope, s->window == 0, ds);
        e |= sm.mark("qkv_dense");
        e |= launch_attn_fwd(dt, QKVd, nullptr, B * Hd, T, dh, causal, s->window, Ad, lsed,
                             at<float>(scratch, L.apart_d), 1, sm.marker(), ds);
        if (ax) {
            e |= launch_out_combine(dt, Ad, w->Wo_d, slot, Xo, B, T, d, H, dh, k, Hd, Y, accumulate,
                                    at<void>(scratch, L.ybase), 1, sm.marker(), ds);
        }
    }
    if (H > 0) {
        if (routed(s)) {
            float* z = at<float>(scratch, L.z);
            float* xnorm = at<float>(scratch, L.xnorm);
            e |= launch_router(dt, X, w->Wr, B, T, d, H, z, xnorm, stream);
            e |= sm.mark("router");
            e |= launch_select(dt, z, xnorm, X, w->Wr, B, T, d, H, k, s->first_token, I, r, slot,
                               at<int32_t>(scratch, L.unc_tok), at<double>(scratch, L.unc_key),
                               at<int32_t>(scratch, L.unc_sel), status, stream);
        } else {
            e |= launch_fixed_select(B, T, H, k, s->fixed_stride, I, r, slot, status, stream);
        }
        e |= sm.mark("select");
        const int fused = launch_qkv_attn(dt, X, I, w->Wq, w->Wk, w->Wv, B, T, d, H, dh, k, QKV, rope, r, causal, A,
                                          lse, stream);
        if (fused == 1) {
            e |= launch_qkv(dt, X, I, w->Wq, w->Wk, w->Wv, B, T, d, H, dh, k, QKV, rope, 0, stream);
            e |= sm.mark("qkv");
            e |= launch_attn_fwd(dt, QKV, r, B * H, k, dh, causal, 0, A, lse, apart, 0, sm.marker(), stream);
        } else {
            e |= fused;
            e |= sm.mark("qkv_attn");
        }
        e |= launch_out_proj(dt, A, w->Wo, B, d, H, dh, k, Xo, stream);
        e |= sm.mark("out_proj");
    }
    if (ax) e |= aux_join(ax, stream);
    e |= launch_out_combine(dt, Ad, w->Wo_d, slot, Xo, B, T, d, H, dh, k, Hd, Y, accumulate,
                            at<void>(scratch, L.ybase), ax ? 2 : 0, sm.marker(), stream);
    if (H > 0 && I_out)
        e |= hipMemcpyAsync(I_out, I, (size_t)B * H * k * 4, hipMemcpyDeviceToDevice, stream) != hipSuccess;
    if (H > 0 && r_out)
        e |= hipMemcpyAsync(r_out, r, (size_t)B * H * k * 4, hipMemcpyDeviceToDevice, stream) != hipSuccess;
    return e ? MOSA_ERR_HIP : MOSA_OK;
}

}  // namespace mosa

extern "C" {

int mosa_forward_timed(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y, int accumulate,
                       int32_t* I_out, float* r_out, void* saved, size_t saved_bytes, void* scratch,
                       size_t scratch_bytes, void* stream, mosa_stage_events* ev) {
    return forward_impl(s, X, w, Y, accumulate, I_out, r_out, saved, saved_bytes, scratch, scratch_bytes, stream, ev,
                        false);
}

int mosa_forward(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y, int accumulate,
                 int32_t* I_out, float* r_out, void* saved, size_t saved_bytes, void* scratch, size_t scratch_bytes,
                 void* stream) {
    return forward_impl(s, X, w, Y, accumulate, I_out, r_out, saved, saved_bytes, scratch, scratch_bytes, stream,
                        nullptr, false);
}

int mosa_backward_timed(const mosa_shape* s, const void* X, const mosa_weights* w, const void* dY, const void* saved,
                        size_t saved_bytes, void* dX, int accumulate_dX, const mosa_grads* g, void* scratch,
                        size_t scratch_bytes, void* stream_, mosa_stage_events* ev) {
    int st = validate_shape(s);
    if (st) return st;
    if ((st = check_weights(s, w))) return st;
    if (!X || !dY || !dX || !g || !aligned(X, 16) || !aligned(dY, 16) || !aligned(dX, 16)) return MOSA_ERR_INVALID_ARG;
    if (!saved || !scratch || !aligned(saved, kAlign) || !aligned(scratch, kAlign)) return MOSA_ERR_INVALID_ARG;
    if (s->heads > 0) {
        const void* need[4] = {g->dWq, g->dWk, g->dWv, g->dWo};
        for (const void* p : need)
            if (!p || !aligned(p, 16)) return MOSA_ERR_INVALID_ARG;
        if ((routed(s) && !g->dWr) || (g->dWr && !aligned(g->dWr, 16))) return MOSA_ERR_INVALID_ARG;
    }
    if (s->dense_heads > 0) {
        const void* need[4] = {g->dWq_d, g->dWk_d, g->dWv_d, g->dWo_d};
        for (const void* p : need)
            if (!p || !aligned(p, 16)) return MOSA_ERR_INVALID_ARG;
    }
    const Layout L = make_layout(s);
    if (saved_bytes < L.saved.total || scratch_bytes < L.scratch_total) return MOSA_ERR_WORKSPACE;

    hipStream_t stream = static_cast<hipStream_t>(stream_);
    if (ev) ev->count = 0;
    StageMarks sm{ev, stream};
    int e = sm.mark("start");
    const int B = s->batch, T = s->seq_len, d = s->d_model, H = s->heads, Hd = s->dense_heads, dh = s->d_head;
    const int k = H > 0 ? s->k : 0, dt = s->dtype, causal = s->causal;
    const int32_t* I = at<int32_t>(saved, L.saved.I);
    const float* r = at<float>(saved, L.saved.r);
    const int16_t* slot = at<int16_t>(saved, L.saved.slot);
    const void* QKV = at<char>(saved, L.saved.QKV);
    const void* A = at<char>(saved, L.saved.A);
    const float* lse = at<float>(saved, L.saved.lse);
    const void* QKVd = at<char>(saved, L.saved.QKVd);
    const void* Ad = at<char>(saved, L.saved.Ad);
    const float* lsed = at<float>(saved, L.saved.lsed);
    void* dA = at<char>(scratch, L.dA);
    float* D = at<float>(scratch, L.D);
    float* dz = at<float>(scratch, L.dz);
    void* dz16 = at<char>(scratch, L.dz16);
    void* dQKV = at<char>(scratch, L.dQKV);
    void* dXs = at<char>(scratch, L.dXs);
    void* dAd = at<char>(scratch, L.dAd);
    float* Dd = at<float>(scratch, L.Dd);
    void* dQKVd = at<char>(scratch, L.dQKVd);
    float* wpart = at<float>(scratch, L.wpart);
    const float2* rope = s->rope ? at<float2>(saved, L.saved.rope) : nullptr;
    // Without a router (fixed sparse attention) r = 1, so dz = dr r (1 - r) = 0
    // and every router term vanishes; W^Q stands in for the unread-in-effect
    // W^r rows (multiplied by dz = 0) and dW^r (all zeros) goes to a sink
    // when the caller passes none.
    const void* Wr = w->Wr ? w->Wr : w->Wq;
    void* dWr = g->dWr ? g->dWr : at<char>(scratch, L.dwr);

    const Marker mk = sm.marker();
    // the dense heads on the auxiliary stream (untimed calls with both kinds of heads)
    std::unique_lock<std::mutex> lock(g_aux_mu, std::defer_lock);
    AuxStream* ax = nullptr;
    if (!ev && H > 0 && Hd > 0 && combine_split_ok(d, H)) {
        lock.lock();
        ax = aux_stream();
        if (ax && aux_fork(ax, stream)) return MOSA_ERR_HIP;
    }
    if (Hd > 0) {
        hipStream_t ds = ax ? ax->s : stream;
        float* wpd = at<float>(scratch, L.wpart_d);
        e |= launch_dattn_out(dt, dY, nullptr, nullptr, w->Wo_d, Ad, B, T, d, Hd, dh, T, dAd, Dd, nullptr, nullptr,
                              ds);
        e |= sm.mark("bwd_out_dense");
        // dW^O needs only dY and the saved A: it goes before the attention
        // backward, so that the chain's tail after it is short
        e |= launch_wgrad(dt, X, dY, nullptr, Ad, dQKVd, nullptr, B, T, d, Hd, dh, T, g->dWq_d, g->dWk_d,
                          g->dWv_d, nullptr, g->dWo_d, wpd, 1, mk, ds);
        e |= launch_attn_bwd(dt, QKVd, dAd, lsed, Dd, B * Hd, T, dh, causal, s->window, dQKVd, nullptr, rope, 1, mk,
                             ds);
        // dQKV of the dense heads is complete: their dX GEMM may start on the
        // main stream once the MoSA heads' kernels are done
        if (ax && hipEventRecord(ax->mid, ds) != hipSuccess) e |= 1;
        e |= launch_wgrad(dt, X, dY, nullptr, Ad, dQKVd, nullptr, B, T, d, Hd, dh, T, g->dWq_d, g->dWk_d,
                          g->dWv_d, nullptr, g->dWo_d, wpd, 0, mk, ds);
    }
    if (H > 0) {
        e |= launch_dattn_out(dt, dY, I, r, w->Wo, A, B, T, d, H, dh, k, dA, D, dz, dz16, stream);
        e |= sm.mark("bwd_out");
        // with the rotary encoding, dQ and dK leave these kernels turned back
        // through the rotation (the gradients of the unrotated q and k)
        e |= launch_attn_bwd(dt, QKV, dA, lse, D, B * H, k, dh, causal, 0, dQKV, I, rope, 0, mk, stream);
        // the weight gradients and the dX rows in one grouped launch where it applies
        const int grouped = launch_bwd_proj(dt, X, dY, I, A, dQKV, dz16, dz, w->Wq, w->Wk, w->Wv, Wr, B, T, d, H, dh,
                                            k, g->dWq, g->dWk, g->dWv, dWr, g->dWo, dXs, stream);
        if (grouped < 0) e |= 1;
        if (grouped == 0) e |= sm.mark("bwd_proj");
        if (grouped == 1) {
            e |= launch_wgrad(dt, X, dY, I, A, dQKV, dz16, B, T, d, H, dh, k, g->dWq, g->dWk, g->dWv, dWr, g->dWo,
                              wpart, 2, mk, stream);
            e |= launch_dx_proj(dt, dQKV, dz, w->Wq, w->Wk, w->Wv, Wr, B, d, H, dh, k, dXs, stream);
            e |= sm.mark("dx_proj");
        }
    }
    if (ax) {
        if (hipStreamWaitEvent(stream, ax->mid, 0) != hipSuccess) e |= 1;
        e |= launch_dx_combine(dt, dQKVd, w->Wq_d, w->Wk_d, w->Wv_d, slot, dXs, B, T, d, H, dh, k, Hd, dX,
                               accumulate_dX, at<void>(scratch, L.dxbase), 1, mk, stream);
    }
    e |= launch_dx_combine(dt, dQKVd, w->Wq_d, w->Wk_d, w->Wv_d, slot, dXs, B, T, d, H, dh, k, Hd, dX, accumulate_dX,
                           at<void>(scratch, L.dxbase), ax ? 2 : 0, mk, stream);
    // nothing on the main stream needs the auxiliary chain's last kernels (the
    // dense heads' dW^{Q,K,V}), so the call's join comes last
    if (ax) e |= aux_join(ax, stream);
    return e ? MOSA_ERR_HIP : MOSA_OK;
}

int mosa_adaptive_k(int seq_len, int rho) {
    if (seq_len < 1 || rho < 1) return 0;
    const int k = seq_len / rho > 2 ? seq_len / rho : 2;
    return k < seq_len ? k : seq_len;
}

int mosa_backward(const mosa_shape* s, const void* X, const mosa_weights* w, const void* dY, const void* saved,
                  size_t saved_bytes, void* dX, int accumulate_dX, const mosa_grads* g, void* scratch,
                  size_t scratch_bytes, void* stream) {
    return mosa_backward_timed(s, X, w, dY, saved, saved_bytes, dX, accumulate_dX, g, scratch, scratch_bytes, stream,
                               nullptr);
}

}  // extern "C"
