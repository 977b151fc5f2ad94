/*
 * mosa.h -- C ABI of the MI355X (gfx950) Mixture of Sparse Attention layer.
 *
 * The layer (paper, Section 2.2 and Eq. 3): every MoSA head h scores all T
 * tokens of a sequence with a sigmoid router r = sigma(X W^r_h), keeps its k
 * highest-scoring tokens I (expert-choice TopK, chosen independently for each
 * batch element), computes Q, K, V only for those tokens, runs attention
 * among them under the index-aware causal mask M_ij = 0 iff I_i >= I_j
 * (Eq. 1), scales output row i by r_{I_i}, projects it with W^O_h and adds it
 * back at position I_i of the T-long output.  The layer output is the sum
 * over heads.  Optional dense heads (the hybrid layer of the "Hybridization"
 * paragraph, standard causal heads of Eq. 2) are added to the same output.
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are DEVICE pointers, row-major, owned by the
 *     caller.  The library allocates no device memory and keeps no data
 *     between calls; temporary memory comes in through `scratch`, state kept
 *     from the forward for the backward through `saved`.  What it does keep
 *     per device: kernels that need more than 64 KB of LDS have that limit set
 *     on the current device before each launch; mosa_forward_noalloc keeps
 *     the address of its static scratch; and the untimed forward and backward
 *     of a layer with both MoSA and dense heads run the dense heads' kernels
 *     on an auxiliary stream of the device (non-blocking, default priority,
 *     created at the first such call and kept until the process ends), forked
 *     from and joined back into `stream` with events inside the call, so the
 *     two sets of heads share the CUs.  The enqueue of such calls is
 *     serialised by a library mutex.  Calls from several host threads, on one
 *     device or several, do not interfere as long as they use different
 *     buffers.
 *   - `stream` is a hipStream_t (NULL: the default stream).  Calls only
 *     enqueue work: everything they enqueue, on the auxiliary stream too, is
 *     complete when work enqueued on `stream` after the call starts, and
 *     errors raised while kernels execute surface at the next synchronisation
 *     of that stream.
 *   - Storage type (`dtype`): MOSA_BF16 or MOSA_F32 for X, dY, every weight,
 *     Y, dX and every weight gradient.  Accumulation is always fp32.
 *     Router logits, r and log-sum-exp values are fp32.
 *   - Every tensor pointer must be 16-byte aligned; `saved` and `scratch`
 *     256-byte aligned.
 *   - Return value: MOSA_OK (0) or a negative status, see mosa_status_string.
 *     Arguments are validated before any work is enqueued; no exception
 *     crosses the ABI.
 *   - Results are bitwise deterministic for identical inputs and shapes,
 *     independent of stream and of the previous contents of scratch.
 *
 * Selection contract (Section 2.2 TopK, read as): the key of token t for
 * head h is the exact value s_t = sum_c X[b,t,c] W^r[h,c] rounded once to
 * double; the k tokens that come first under (key descending, token index
 * ascending) are selected -- ties go to the lower index -- and I is returned
 * in ascending order.  sigma is strictly increasing, so this is the TopK of
 * r.  r_i = sigma(s_{I_i}) is computed in fp32 from the fp32 logit.
 */
#ifndef MOSA_H
#define MOSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    MOSA_OK = 0,
    MOSA_ERR_INVALID_ARG = -1, /* bad size, null required pointer, misalignment */
    MOSA_ERR_UNSUPPORTED = -2, /* valid but not implemented (d_head, d_model, T range) */
    MOSA_ERR_WORKSPACE = -3,   /* saved or scratch smaller than mosa_workspace_size */
    MOSA_ERR_HIP = -4          /* a HIP launch or query failed */
};

typedef enum { MOSA_F32 = 0, MOSA_BF16 = 1 } mosa_dtype;

/* Shape of one layer call.  Limits: batch >= 1; 1 <= seq_len <= 16384;
 * d_model a multiple of 64; d_head 32 or 64; heads >= 0 and dense_heads >= 0
 * with heads + dense_heads >= 1; 1 <= k <= seq_len when heads > 0
 * (k = seq_len selects every token); causal 0 or 1.
 *
 * Variants of the layer (0 = off; a zero-initialised tail gives the plain
 * layer):
 *   first_token   1: every MoSA head always keeps token 0 and chooses the
 *                 other k - 1 among t >= 1 by router score; token 0 is scaled
 *                 by its own r (Section 3.2, IsoFLOP setting).
 *   fixed_stride  rho > 0: fixed sparse attention as a special case of MoSA
 *                 (Section 3.1): I = 0, rho, ..., (k - 1) rho for every head
 *                 and batch element, r = 1, no router.  Needs
 *                 (k - 1) rho <= seq_len - 1 and first_token == 0; W^r may be
 *                 NULL in mosa_forward / mosa_backward and dW^r NULL in
 *                 mosa_backward (when given it is written with zeros).
 *   rope          1: rotary position encoding of q and k after the
 *                 projections, at the tokens' ORIGINAL positions I
 *                 (Section 2.2, "Positional encodings"); dense heads use
 *                 positions 0..T-1.  The first d_head/2 dimensions are rotated
 *                 in adjacent pairs (2j, 2j+1) by the angle
 *                 p * rope_base^(-2j/(d_head/2)); the other half is unchanged.
 *   rope_base     the base of those angles (> 1; used when rope == 1).
 *   window        w > 0: the dense heads are local (sliding-window) causal
 *                 heads, query t seeing keys t - w + 1 .. t (Section 3.4);
 *                 needs causal == 1. */
typedef struct mosa_shape {
    int32_t batch;       /* B */
    int32_t seq_len;     /* T */
    int32_t d_model;     /* d, the paper's h */
    int32_t heads;       /* H, MoSA heads */
    int32_t d_head;      /* dh, the paper's h' */
    int32_t k;           /* tokens kept per MoSA head and batch element */
    int32_t causal;      /* 1: M_ij = 0 iff I_i >= I_j; 0: no mask */
    int32_t dense_heads; /* Hd, dense heads (all T tokens, r = 1) */
    int32_t dtype;       /* mosa_dtype */
    int32_t first_token; /* variants, see above */
    int32_t fixed_stride;
    int32_t rope;
    float rope_base;
    int32_t window;
} mosa_shape;

/* The paper's adaptive k for short inputs (Section 3.5): max(floor(T / rho), 2),
 * clamped to T; rho >= 1. Returns 0 for invalid arguments. */
int mosa_adaptive_k(int seq_len, int rho);

/* Layer parameters, theta_h = (W^Q, W^K, W^V, W^O, W^r) per head (Section 2.2),
 * in the paper's X W orientation:
 *   Wr [H, d]; Wq, Wk, Wv [H, d, dh]; Wo [H, dh, d];
 *   dense heads: Wq_d, Wk_d, Wv_d [Hd, d, dh]; Wo_d [Hd, dh, d] (NULL iff Hd == 0). */
typedef struct mosa_weights {
    const void* Wr;
    const void* Wq;
    const void* Wk;
    const void* Wv;
    const void* Wo;
    const void* Wq_d;
    const void* Wk_d;
    const void* Wv_d;
    const void* Wo_d;
} mosa_weights;

/* Weight gradients, same shapes and storage type as mosa_weights; written
 * (not accumulated).  Dense entries NULL iff Hd == 0. */
typedef struct mosa_grads {
    void* dWr;
    void* dWq;
    void* dWk;
    void* dWv;
    void* dWo;
    void* dWq_d;
    void* dWk_d;
    void* dWv_d;
    void* dWo_d;
} mosa_grads;

/* Byte offsets of the tensors the forward leaves in `saved` (read-only for
 * the caller; documented so that tests can inspect the stages):
 *   I [B,H,k] int32 ascending; r [B,H,k] fp32;
 *   slot [B,H,T] int16: position of token t in I[b,h,:], or -1;
 *   QKV [B,H,k,3,dh] storage type: packed rows q | k | v of the selected tokens;
 *   A [B,H,k,dh] storage type (attention output rows already scaled by the
 *     router value: r_i (softmax(Q K^T / sqrt(dh) + M) V)_i);
 *   lse [B,H,k] fp32 (natural-log sum of exp of the scaled scores);
 *   the same for the dense heads with k = T: QKVd [B,Hd,T,3,dh], Ad [B,Hd,T,dh],
 *   lsed [B,Hd,T];
 *   rope [T, dh/4] float2 (cos, sin) table of the rotary encoding (rope == 1);
 *   status [B,H] int32: 0 when the selection of row (b, h) holds exactly k
 *     certified tokens; 1 when it does not, which happens only if the
 *     router's logit error bound (an assumption about the MFMA adder, see
 *     mosa_forward) failed: I and r of that row are then padded with token 0
 *     and r = 0 or cut at k, and the outputs of the call must not be used.
 *     Callers that need the guarantee read this array after the forward. */
typedef struct mosa_saved_layout {
    size_t I, r, slot, QKV, A, lse, QKVd, Ad, lsed, rope, status;
    size_t total;
} mosa_saved_layout;

/* Sizes in bytes of the two caller-provided buffers for shape `s`:
 * `saved` (written by mosa_forward, read by mosa_backward) and `scratch`
 * (temporary; large enough for both forward and backward). */
int mosa_workspace_size(const mosa_shape* s, size_t* saved_bytes, size_t* scratch_bytes);

/* Offsets of the saved tensors (see mosa_saved_layout). */
int mosa_saved_offsets(const mosa_shape* s, mosa_saved_layout* out);

/* Forward of the layer (Section 2.2, Eq. 1-3).
 *   X [B,T,d]; Y [B,T,d]: Y = layer(X) if accumulate == 0, Y += layer(X)
 *   otherwise (residual stream).  Rows of Y no head selects and no dense head
 *   covers are exactly 0 (accumulate == 0) or unchanged.
 *   I_out [B,H,k] int32, r_out [B,H,k] fp32: optional copies of the
 *   selection (NULL to skip).
 *   saved / scratch: caller buffers of at least the mosa_workspace_size
 *   sizes; `saved` must stay unmodified until the matching mosa_backward.
 *   When H > 0, the first B*H*T*4 bytes of `scratch` hold the fp32 router
 *   logits z [B,H,T] after the call (until scratch is reused).
 *   The selection is certified against the exact keys with an error bound
 *   on the fp32 router logits that assumes each 32-term MFMA chunk sum lies
 *   within (K+1) units in the last place of its largest term of the exact
 *   chunk sum (doubled for margin); the selection status in `saved` records
 *   any row where that assumption failed. */
int mosa_forward(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y,
                 int accumulate, int32_t* I_out, float* r_out, void* saved, size_t saved_bytes,
                 void* scratch, size_t scratch_bytes, void* stream);

/* Backward of the layer with the selection I held fixed (TopK is piecewise
 * constant; the router receives its gradient through r, Section 2.2 final
 * paragraph).  dY [B,T,d]; X and w must be the forward's; `saved` the
 * forward's.  dX [B,T,d]: written (accumulate_dX == 0) or added to.
 * All weight gradients in `g` are written. */
int mosa_backward(const mosa_shape* s, const void* X, const mosa_weights* w, const void* dY,
                  const void* saved, size_t saved_bytes, void* dX, int accumulate_dX,
                  const mosa_grads* g, void* scratch, size_t scratch_bytes, void* stream);

/* Stage timing for profiling and benchmarks.  The caller creates up to
 * MOSA_MAX_STAGES hipEvent_t handles and stores them in `events`; the timed
 * variants below launch exactly the kernels of mosa_forward / mosa_backward,
 * with the same arguments, all on `stream` in one serial order (the dense
 * heads' kernels are not moved to the auxiliary stream), and in addition record
 * events[0] on `stream` before the first kernel and events[j] after the j-th
 * kernel launch, setting names[j] to that kernel's static stage name and
 * `count` to the number of events recorded.  The time of stage j is
 * hipEventElapsedTime(events[j-1], events[j]).  A NULL `ev` makes them
 * identical to the untimed calls. */
#define MOSA_MAX_STAGES 32
typedef struct mosa_stage_events {
    void* events[MOSA_MAX_STAGES];
    const char* names[MOSA_MAX_STAGES];
    int count;
} mosa_stage_events;

int mosa_forward_timed(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y,
                       int accumulate, int32_t* I_out, float* r_out, void* saved,
                       size_t saved_bytes, void* scratch, size_t scratch_bytes, void* stream,
                       mosa_stage_events* ev);
int mosa_backward_timed(const mosa_shape* s, const void* X, const mosa_weights* w, const void* dY,
                        const void* saved, size_t saved_bytes, void* dX, int accumulate_dX,
                        const mosa_grads* g, void* scratch, size_t scratch_bytes, void* stream,
                        mosa_stage_events* ev);

/* Allocation-free forward, for callers that cannot allocate device memory
 * (code under stream capture, tight serving loops, harnesses that forbid
 * hipMalloc): mosa_forward without the `scratch` argument.  Its temporary
 * memory is a static device array of MOSA_NOALLOC_SCRATCH_MAX bytes inside the
 * library, one per GPU, held from the first call on that GPU until the process
 * ends; the call itself allocates nothing.  Shapes whose forward needs more
 * scratch than that are rejected with MOSA_ERR_WORKSPACE before any work is
 * enqueued (the forward's scratch is at most the mosa_workspace_size scratch
 * size: 64 MiB holds, e.g., B=8, T=1024, d_model=512, 32 heads, k=128).  Every call on one GPU uses
 * the same array: calls that overlap in time on one GPU (different streams,
 * or host threads without ordering) race and must be serialised by the
 * caller; consecutive calls on one stream are safe.  Nothing in the array
 * needs clearing between calls (every byte the forward reads there it first
 * wrote in the same call).  The library keeps the array's per-device address
 * from the first call on each device.  Results equal mosa_forward's bit for
 * bit. */
#define MOSA_NOALLOC_SCRATCH_MAX ((size_t)64 << 20)
int mosa_forward_noalloc(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y, int accumulate,
                         int32_t* I_out, float* r_out, void* saved, size_t saved_bytes, void* stream);

/* Static text for a status code (never NULL). */
const char* mosa_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* MOSA_H */
