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
constexpr int kSegWidth = 64;  // token width of one entry of the per-head segment table

inline int seg_count(int T) { return (T + kSegWidth - 1) / kSegWidth + 1; }

// z[b,h,t] = X[b,t,:] . Wr[h,:] (fp32), xnorm[b*T+t] >= ||X[b,t,:]||_2.
int launch_router(int dtype, const void* X, const void* Wr, int B, int T, int d, int H, float* z,
                  float* xnorm, hipStream_t stream);

// Certified expert-choice top-k per (b,h): I ascending, r = sigmoid(z) at I,
// seg[b,h,j] = #selected tokens < 64 j.  unc_tok / unc_key / unc_sel are
// per-row scratch of T entries each.
int launch_select(int dtype, const float* z, const float* xnorm, const void* X, const void* Wr, int B,
                  int T, int d, int H, int k, int32_t* I, float* r, int32_t* seg, int32_t* unc_tok,
                  double* unc_key, int32_t* unc_sel, hipStream_t stream);

// out_{q,k,v}[b,h,i,:] = X[b, I[b,h,i], :] . W_{q,k,v}[h]  for i < n
// (I == nullptr: identity, i.e. a dense head with n = T).
int launch_qkv(int dtype, const void* X, const int32_t* I, const void* Wq, const void* Wk,
               const void* Wv, int B, int T, int d, int H, int dh, int n, void* Q, void* K, void* V,
               hipStream_t stream);

// A = softmax(Q K^T / sqrt(dh) + causal mask in slot order) V per (b,h);
// lse = log-sum-exp of the scaled scores (natural log).
int launch_attn_fwd(int dtype, const void* Q, const void* K, const void* V, int BH, int n, int dh,
                    int causal, void* A, float* lse, hipStream_t stream);

// Y[b,t,:] (+)= sum_h sum_{i: I[b,h,i]=t} r[b,h,i] A[b,h,i,:] Wo[h]
//              + sum_hd Ad[b,hd,t,:] Wo_d[hd], heads in a fixed order.
int launch_out_scatter(int dtype, int B, int T, int d, int dh, int H, int k, const int32_t* I,
                       const float* r, const int32_t* seg, const void* A, const void* Wo, int Hd,
                       const void* Ad, const void* Wo_d, void* Y, int accumulate, hipStream_t stream);

// Backward, output side of a head: dA~ = dY[I] Wo^T; dA = r dA~;
// D = r <dA~, A>; dz = <dA~, A> r (1 - r) (dz may be null: dense heads, r null).
int launch_dattn_out(int dtype, const void* dY, const int32_t* I, const float* r, const void* Wo, const void* A,
                     int B, int T, int d, int H, int dh, int n, void* dA, float* D, float* dz, hipStream_t stream);

// Attention backward; pass 0 writes dK, dV, pass 1 writes dQ.
int launch_attn_bwd(int dtype, const void* Q, const void* K, const void* V, const void* dA, const float* lse,
                    const float* D, int BH, int n, int dh, int causal, void* dQ, void* dK, void* dV, int pass,
                    hipStream_t stream);

// Weight gradients; which 0: dWq, dWk, dWv (+ dWr when non-null), which 1: dWo.
int launch_wgrad(int dtype, const void* X, const void* dY, const int32_t* I, const float* r, const void* A,
                 const void* dQ, const void* dK, const void* dV, const float* dz, int B, int T, int d, int H, int dh,
                 int n, void* dWq, void* dWk, void* dWv, void* dWr, void* dWo, int which, hipStream_t stream);

// dX[b,t,:] (+)= sum_h sum_{i: I=t} (dQ Wq^T + dK Wk^T + dV Wv^T + dz Wr)_i + dense heads.
int launch_dx_scatter(int dtype, int B, int T, int d, int dh, int H, int k, const int32_t* I, const int32_t* seg,
                      const void* dQ, const void* dK, const void* dV, const float* dz, const void* Wq, const void* Wk,
                      const void* Wv, const void* Wr, int Hd, const void* dQd, const void* dKd, const void* dVd,
                      const void* Wq_d, const void* Wk_d, const void* Wv_d, void* dX, int accumulate,
                      hipStream_t stream);

}  // namespace mosa
