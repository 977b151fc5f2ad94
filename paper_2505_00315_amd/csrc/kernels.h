// Internal launch functions of the MoSA kernels (not part of the C ABI).
// Every launcher enqueues on `stream`, returns 0 on success and -1 when the
// launch itself failed.  Shapes have been validated by the host layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mosa {

constexpr int kF32 = 0;
constexpr int kBF16 = 1;

// Stage hook of the timed entry points: launchers that enqueue more than one
// kernel call it after each of them with that kernel's stage name (a static
// string), so that an event can be recorded between any two launches.  A
// default-constructed Marker does nothing.
struct Marker {
    int (*fn)(void* ctx, const char* name) = nullptr;
    void* ctx = nullptr;
    int operator()(const char* name) const { return fn ? fn(ctx, name) : 0; }
};

// z[b,h,t] = X[b,t,:] . Wr[h,:] (fp32), xnorm[b*T+t] >= ||X[b,t,:]||_2.
int launch_router(int dtype, const void* X, const void* Wr, int B, int T, int d, int H, float* z,
                  float* xnorm, hipStream_t stream);

// Certified expert-choice top-k per (b,h): I ascending, r = sigmoid(z) at I,
// slot[b,h,t] = position of t in I or -1.  unc_tok / unc_key / unc_sel are
// per-row scratch of T entries each.
// first_token: token 0 is always kept, the other k - 1 chosen among t >= 1.
// status[b,h] = 0 when exactly k tokens were certified, else 1 (the logit
// error bound failed; I is then padded or cut and must not be used).
int launch_select(int dtype, const float* z, const float* xnorm, const void* X, const void* Wr, int B,
                  int T, int d, int H, int k, int first_token, int32_t* I, float* r, int16_t* slot,
                  int32_t* unc_tok, double* unc_key, int32_t* unc_sel, int32_t* status, hipStream_t stream);

// Fixed sparse attention (no router): I[b,h,i] = i * stride, r = 1, the slot
// map, and status = 0.
int launch_fixed_select(int B, int T, int H, int k, int stride, int32_t* I, float* r, int16_t* slot,
                        int32_t* status, hipStream_t stream);

// Rotary encoding: tab [T, dh/4] (cos, sin) pairs of positions 0..T-1.
int launch_rope_table(int T, int dh, float base, float2* tab, hipStream_t stream);

// QKV[b,h,i,:] = X[b, I[b,h,i], :] . [Wq | Wk | Wv][h]  (packed rows of 3*dh)
// for i < n (I == nullptr: identity, i.e. a dense head with n = T); with a
// rotary table, q and k rotated at position I[b,h,i] (or i).  narrow: tiles
// of 64 rows instead of 128 (bf16).
int launch_qkv(int dtype, const void* X, const int32_t* I, const void* Wq, const void* Wk,
               const void* Wv, int B, int T, int d, int H, int dh, int n, void* QKV, const float2* rope,
               int narrow, hipStream_t stream);

// A = diag(r) softmax(Q K^T / sqrt(dh) + causal mask in slot order) V per
// (b,h) (r == nullptr: r = 1); lse = log-sum-exp of the scaled scores
// (natural log).
// Q/K/V projection and attention in one launch for bf16 groups of
// n = 16, 32, 64 or 128 rows (the outputs of launch_qkv and launch_attn_fwd);
// returns 1 without launching when the shape does not qualify.
int launch_qkv_attn(int dtype, const void* X, const int32_t* I, const void* Wq, const void* Wk, const void* Wv,
                    int B, int T, int d, int H, int dh, int n, void* QKV, const float2* rope, const float* r,
                    int causal, void* A, float* lse, hipStream_t stream);
// window > 0 (causal only): query t sees keys t - window + 1 .. t (local heads).
// part: fp32 scratch of attn_fwd_part_bytes(...) bytes for the partial
// results of long query blocks cut into key splits (nullptr when that is 0).
// Marks "attn" (dense heads: "attn_dense"), and "attn_merge" /
// "attn_dense_merge" after the kernel that combines the splits.
int launch_attn_fwd(int dtype, const void* QKV, const float* r, int BH, int n, int dh, int causal, int window, void* A,
                    float* lse, float* part, int dense, const Marker& mk, hipStream_t stream);
size_t attn_fwd_part_bytes(int dtype, int BH, int n, int dh, int causal, int window);

// Xo[b,h,i,:] = A[b,h,i,:] Wo[h]  (A already scaled by r).
int launch_out_proj(int dtype, const void* A, const void* Wo, int B, int d, int H, int dh, int k, void* Xo,
                    hipStream_t stream);

// Y[b,t,:] (+)= sum_hd Ad[b,hd,t,:] Wo_d[hd] + sum_h (ascending) Xo[b,h,slot[b,h,t],:].
// base: [B, T, d] scratch in the storage type for the dense heads' part (used
// when Hd > 0).  Marks "out_dense" (the dense heads' GEMM, when launched separately) and
// "out_combine".  part 1: only the dense heads' GEMM into base, part 2: only
// the combination (base written before), 0: both; parts 1 and 2 need
// combine_split_ok(d, H) (else they return 1 and launch nothing).
int launch_out_combine(int dtype, const void* Ad, const void* Wo_d, const int16_t* slot, const void* Xo,
                       int B, int T, int d, int H, int dh, int k, int Hd, void* Y, int accumulate, void* base,
                       int part, const Marker& mk, hipStream_t stream);
bool combine_split_ok(int d, int H);

// Backward, output side of a head (A is the r-scaled attention output):
// dA~ = dY[I] Wo^T; dA = r dA~; D = <dA~, A>; dz = D (1 - r) (also as 16-wide
// rows dz16); dz, dz16 may be null and I, r null for dense heads.
int launch_dattn_out(int dtype, const void* dY, const int32_t* I, const float* r, const void* Wo,
                     const void* A, int B, int T, int d, int H, int dh, int n, void* dA, float* D, float* dz,
                     void* dz16, hipStream_t stream);

// Attention backward into packed dQKV rows (dQ, dK and dV; one launch where
// the kernels allow it).  Marks "attn_bwd" (dense heads: "attn_bwd_dense"),
// or "attn_bwd_kv" and "attn_bwd_q" (+ "_dense") when the passes are two
// launches.
int launch_attn_bwd(int dtype, const void* QKV, const void* dA, const float* lse, const float* D, int BH,
                    int n, int dh, int causal, int window, void* dQKV, const int32_t* rope_I,
                    const float2* rope, int dense, const Marker& mk, hipStream_t stream);

// Weight gradients; which 0: dWq, dWk, dWv (+ dWr when non-null), which 1: dWo,
// which 2: both (in one launch where the gathered-row engine applies).
// part: fp32 scratch of wgrad_partial_bytes(...) bytes for split row ranges.
// Marks every kernel: "wgrad" (both in one launch), else "wgrad_qkv" and
// "wgrad_o", each followed by "<name>_reduce" where partials are summed;
// dense heads (I == nullptr) the same names with "_dense".
int launch_wgrad(int dtype, const void* X, const void* dY, const int32_t* I, const void* A,
                 const void* dQKV, const void* dz16, int B, int T, int d, int H, int dh, int n, void* dWq,
                 void* dWk, void* dWv, void* dWr, void* dWo, float* part, int which, const Marker& mk,
                 hipStream_t stream);
size_t wgrad_partial_bytes(int dtype, int B, int d, int H, int dh, int n, int router);
// The MoSA heads' dW^{Q,K,V,r}, dW^O and per-head dX rows (launch_dx_proj) in
// one grouped launch; returns 1, launching nothing, where that does not apply.
int launch_bwd_proj(int dtype, const void* X, const void* dY, const int32_t* I, const void* A, const void* dQKV,
                    const void* dz16, const float* dz, const void* Wq, const void* Wk, const void* Wv, const void* Wr,
                    int B, int T, int d, int H, int dh, int n, void* dWq, void* dWk, void* dWv, void* dWr, void* dWo,
                    void* dXs, hipStream_t stream);

// The same three products for heads with at most 128 selected rows over the
// batch (B k <= 128; bf16, 64-wide heads): one workgroup per (product, head,
// range of 64-column tiles of d) with the head's fixed operand in registers and
// the other streamed through LDS; returns 1, launching nothing, where that does
// not apply.
int launch_bwd_head(int dtype, const void* X, const void* dY, const int32_t* I, const void* A, const void* dQKV,
                    const void* dz16, const float* dz, const void* Wq, const void* Wk, const void* Wv, const void* Wr,
                    int B, int T, int d, int H, int dh, int k, void* dWq, void* dWk, void* dWv, void* dWr, void* dWo,
                    void* dXs, hipStream_t stream);

// dXs[b,h,i,:] = dQ Wq^T + dK Wk^T + dV Wv^T + dz Wr  (per selected row).
int launch_dx_proj(int dtype, const void* dQKV, const float* dz, const void* Wq, const void* Wk,
                   const void* Wv, const void* Wr, int B, int d, int H, int dh, int k, void* dXs,
                   hipStream_t stream);

// dX[b,t,:] (+)= dense heads' (dQ Wq^T + dK Wk^T + dV Wv^T) + sum_h (ascending) dXs[b,h,slot,:].
// base: [B, T, d] scratch in the storage type for the dense heads' part (used
// when Hd > 0).  Marks "dx_dense" (when launched separately) and "dx_combine"; part as in
// launch_out_combine.
int launch_dx_combine(int dtype, const void* dQKVd, const void* Wq_d, const void* Wk_d, const void* Wv_d,
                      const int16_t* slot, const void* dXs, int B, int T, int d, int H, int dh, int k,
                      int Hd, void* dX, int accumulate, void* base, int part, const Marker& mk, hipStream_t stream);

}  // namespace mosa
