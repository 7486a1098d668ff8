/*
 * moa_attn.h -- C ABI of the fused scaled dot-product attention library for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation is the paper's problem statement (Sec. "MoA DNF Derivation of
 * Attention", eq. attention with the stable softmax of eq. stable_softmax),
 * applied independently to every (batch, head) slice as the remark on
 * higher-rank tensors in that section prescribes:
 *
 *   O[b,h,i,:] = sum_j P[b,h,i,j] * V[b,h,j,:]
 *   P[b,h,i,:] = softmax over visible j of  scale * <Q[b,h,i,:], K[b,h,j,:]>
 *
 * computed as in the Denotational Normal Form (eqs. dnf_attn, output_dnf):
 * no transposed-K buffer, no score matrix and no softmax temporary is ever
 * written to device memory.  The only device-memory writes of a prefill call
 * are O (and LSE when requested); a call that splits its keys across
 * workgroups (decode, Nq == 1; prefill on grids too small to fill the GPU)
 * additionally writes per-split partial results of size
 * O(B*H*Nq*splits*dv) into the caller's workspace.
 *
 * Conventions shared by all entry points
 *  - Plain C types only; no HIP or framework types appear here.  `stream` is a
 *    hipStream_t passed as void* (NULL = the default stream).
 *  - All tensor pointers are DEVICE pointers owned by the caller.  moa_attn_fwd
 *    takes contiguous row-major tensors (last index fastest; the paper's gamma
 *    layout; moa_attn_fwd_strided below takes per-dimension strides):
 *      Q [B][H][Nq][dk]   K [B][H][Nk][dk]   V [B][H][Nk][dv]   O [B][H][Nq][dv]
 *      LSE [B][H][Nq] fp32 (optional, NULL = not written)
 *    Every tensor pointer must be 16-byte aligned.
 *  - The library allocates no device memory, keeps no state between calls,
 *    never synchronises, and is safe to call from several host threads (the
 *    one exception: moa_attn_fwd_noalloc's fixed scratch array, below).  Work
 *    is enqueued on `stream` (at most two kernels for the forward, three for
 *    the projected forward and for the backward); errors raised by kernels
 *    surface at the caller's next synchronisation.
 *  - Arguments are validated on the host before any HIP call; a rejected call
 *    touches no device memory.
 */
#ifndef MOA_ATTN_H
#define MOA_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
enum {
    MOA_OK = 0,
    MOA_ERR_INVALID_ARG = 1,  /* NULL pointer, bad dimension, misaligned or overlapping buffers,
                                 non-finite scale, causal with Nq > Nk, unknown dtype */
    MOA_ERR_UNSUPPORTED = 2,  /* valid request this build does not implement (head size) */
    MOA_ERR_WORKSPACE = 3,    /* workspace missing or smaller than moa_attn_workspace_bytes() */
    MOA_ERR_HIP = 4,          /* the HIP runtime reported an error while enqueueing */
    MOA_ERR_SCRATCH = 5       /* moa_attn_fwd_noalloc: the call needs more scratch than the
                                 library's fixed array holds (MOA_NOALLOC_SCRATCH_BYTES) */
};

/* Storage types for Q, K, V (in_dtype) and O (out_dtype). */
enum {
    MOA_F32 = 0,   /* IEEE binary32 */
    MOA_BF16 = 1   /* bfloat16 (upper half of binary32) */
};

/*
 * moa_attn_workspace_bytes -- device workspace a moa_attn_fwd call with the
 * same arguments needs, in bytes (0 when none).
 *
 * Calls that split the key range into chunks (`num_splits`; 0 = the
 * library's choice, which this function then reports for) and combine the
 * partial softmax results in a second pass need a workspace for those
 * partials: B*H*Nq*splits rows of dv + 2 fp32 values, rounded up to 256
 * bytes.  Decode-shaped calls (Nq == 1) split when the library's choice (or
 * `num_splits` > 1) says so: automatically so that B*H*splits reaches about
 * 256 workgroups with at least 256 keys per split; with one split the call
 * writes O directly and needs no workspace.  bf16 prefill calls
 * (Nq > 1) split when the library's choice (or `num_splits` > 1) says so:
 * automatically only for grids too small to fill the GPU (fewer than 128
 * tiles of 256 queries over all B*H slices, and at least 2048 keys), where
 * splits * (128-query tiles) approaches 256 workgroups with at least 1024
 * keys per split.  fp32 prefill never splits (its call ignores the
 * workspace).  Returns 0 when the call does not split and for invalid
 * dimensions.
 */
size_t moa_attn_workspace_bytes(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk,
                                int64_t dv, int num_splits);

/*
 * moa_attn_num_splits -- the number of key splits a call with these
 * arguments will use when given moa_attn_workspace_bytes(...) of workspace
 * (decode-shaped calls, and bf16 prefill; 1 = no split).
 */
int moa_attn_num_splits(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                        int num_splits);

/*
 * moa_attn_fwd -- fused attention forward (eq. attention; DNF eqs. dnf_attn
 * and output_dnf; the max-subtracted softmax of eq. stable_softmax).
 *
 * Q, K, V   device inputs of storage type in_dtype (MOA_F32 or MOA_BF16, the
 *           same for all three), layouts above.
 * O         device output of storage type out_dtype (MOA_F32, or in_dtype).
 * LSE       optional device output, fp32 [B][H][Nq]: the natural log of the
 *           softmax denominator, LSE = max_j s_j + ln(sum_j exp(s_j - max_j s_j))
 *           with s_j = scale * <q, k_j> over visible j.  NULL = not written.
 * B, H      batch and head counts (>= 0).
 * Nq, Nk    query and key counts (Nq >= 0, Nk >= 1).
 * dk, dv    head sizes; supported: dk == dv in {64, 128}.
 * scale     finite fp32 multiplier of the inner products (the paper divides
 *           by sqrt(dk): pass 1/sqrt(dk) for that).  0 and negative values
 *           are valid.
 * causal    0: every key is visible.  1: key j is visible to query i iff
 *           j <= i + (Nk - Nq) (bottom-right aligned; j <= i when Nq == Nk).
 *           Requires Nq <= Nk, so no query row is fully masked.
 * workspace, workspace_bytes
 *           device scratch for calls that split their keys; at least
 *           moa_attn_workspace_bytes(...) bytes, 16-byte aligned, not
 *           overlapping any tensor.  Required for decode-shaped calls that
 *           split and for bf16 prefill with num_splits > 1 (else
 *           MOA_ERR_WORKSPACE);
 *           a bf16 prefill call with num_splits == 0 whose workspace is
 *           missing or too small runs in one pass instead.  May be NULL/0
 *           when moa_attn_workspace_bytes(...) is 0.
 * num_splits
 *           key splits across workgroups (0 = library's choice, else
 *           1..256; 1 = no split).  Ignored by fp32 prefill.
 * stream    hipStream_t as void*.
 *
 * Computation: inner products and softmax statistics in fp32 from exact
 * products of the inputs; bf16 inputs use bf16 matrix-core products with fp32
 * accumulation and the unnormalised weights rounded to bf16 before they
 * multiply V.  For bf16 prefill the denominator is the sum of those same
 * rounded weights, so O is an exact convex combination of V rows with weights
 * within 2^-8 (relative) of the softmax, and LSE is within ln(1 + 2^-8) of the
 * exact value; fp32 inputs and decode-shaped calls keep fp32 weights
 * throughout.  Results are deterministic: identical inputs give bit-identical
 * outputs (no atomics).
 *
 * Returns MOA_OK once the work is enqueued (or when B*H*Nq == 0: nothing is
 * launched), else one of the MOA_ERR_* codes above.
 */
int moa_attn_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE, int64_t B,
                 int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv, float scale, int causal,
                 int in_dtype, int out_dtype, void* workspace, size_t workspace_bytes,
                 int num_splits, void* stream);

/*
 * moa_attn_fwd_strided -- moa_attn_fwd on strided tensors: the storage
 * functions of the footnote to eq. gamma with per-dimension strides, i.e.
 * the Operational Normal Form's offset = base + sum_k stride_k * i_k
 * (Def. "Operational Normal Form").  Element (b, h, i, e) of Q lives at
 *   Q + (b*q_strides[0] + h*q_strides[1] + i*q_strides[2] + e) elements,
 * and likewise for K, V and O; the head dimension e is contiguous.  This
 * covers the row-major [B][H][N][d] layout, [B][N][H][d] (PyTorch's usual
 * batch-first layout without a copy), padded rows, packed QKV buffers, and
 * K/V shared across heads (head stride 0).  A stride array may be NULL, which
 * means the contiguous row-major strides of moa_attn_fwd.  LSE stays
 * contiguous [B][H][Nq].  Column-major storage (non-contiguous e) goes
 * through moa_attn_fwd_onf instead.
 *
 * Stride rules (elements, each array {batch, head, row}):
 *  - all >= 0 (else MOA_ERR_INVALID_ARG); rows of a tensor with more than one
 *    row must not overlap (row stride >= d, else MOA_ERR_INVALID_ARG);
 *  - stride * element size a multiple of 16 bytes, and (rows-1)*row stride + d
 *    elements within 2^31 bytes per head (else MOA_ERR_UNSUPPORTED);
 *  - O must not write any element twice (its dimensions of size > 1, ordered
 *    by stride, must nest without overlap; else MOA_ERR_INVALID_ARG).
 * Q, K and V may overlap one another (they are only read); O, LSE and the
 * workspace must not overlap anything, where a strided tensor occupies the
 * bytes from its base pointer to the end of its last element.
 * All other arguments, results and status codes are those of moa_attn_fwd.
 */
int moa_attn_fwd_strided(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                         const int64_t* q_strides, const int64_t* k_strides,
                         const int64_t* v_strides, const int64_t* o_strides, float scale,
                         int causal, int in_dtype, int out_dtype, void* workspace,
                         size_t workspace_bytes, int num_splits, void* stream);

/*
 * moa_attn_fwd_onf -- moa_attn_fwd on tensors with a stride for EVERY
 * dimension, the head elements included: the storage functions of the
 * footnote to eq. gamma in full generality, every access at
 * offset = base + sum_k stride_k * i_k (Def. "Operational Normal Form").
 * Element (b, h, i, e) of Q lives at
 *   Q + (b*q_strides[0] + h*q_strides[1] + i*q_strides[2] + e*q_strides[3])
 * elements, and likewise for K, V and O.  This covers column-major heads
 * ([B][H][d][N] storage: row stride 1, element stride N), rows that are not
 * 16-byte aligned, rows that overlap (inputs only), and every layout of
 * moa_attn_fwd_strided (element stride 1).  A stride array may be NULL: the
 * contiguous row-major strides.  LSE stays contiguous [B][H][Nq].
 *
 * Dispatch: when every tensor has element stride 1 and meets the stride and
 * alignment rules of moa_attn_fwd_strided, the call is exactly that entry
 * point's (same kernels, workspace and split rules).  Otherwise an
 * element-gather kernel serves it: it reads each element at its own address,
 * computes in fp32 (fp32 or bf16 inputs; fp32 products, exact online
 * softmax), needs no workspace (workspace, workspace_bytes and num_splits are
 * then ignored), and runs far below the matrix-core kernels' throughput.
 *
 * Rules for the gather path: all strides >= 0 (else MOA_ERR_INVALID_ARG);
 * Q, K, V aligned to their element size, O to its element size, LSE to 4
 * bytes; O must not write any element twice (its dimensions of size > 1,
 * ordered by stride, must nest without overlap); O and LSE must not overlap
 * any tensor, a tensor occupying the bytes from its base pointer to its last
 * element.  Q, K and V may overlap one another and themselves.  All other
 * arguments, results and status codes are those of moa_attn_fwd.
 */
int moa_attn_fwd_onf(const void* Q, const void* K, const void* V, void* O, float* LSE,
                     int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                     const int64_t* q_strides, const int64_t* k_strides, const int64_t* v_strides,
                     const int64_t* o_strides, float scale, int causal, int in_dtype,
                     int out_dtype, void* workspace, size_t workspace_bytes, int num_splits,
                     void* stream);

/* Bytes of the fixed device scratch array of moa_attn_fwd_noalloc, per GPU. */
#define MOA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/*
 * moa_attn_fwd_noalloc -- moa_attn_fwd for callers that cannot allocate device
 * memory: code being captured into a HIP graph, tight serving loops, and
 * hosts that forbid allocation.  The arguments, results and status codes are
 * those of moa_attn_fwd without the workspace: the partial states of calls
 * that split their keys (decode-shaped calls; bf16 prefill on grids too small
 * to fill the GPU) go to a fixed scratch array in device memory that the
 * library itself holds, MOA_NOALLOC_SCRATCH_BYTES bytes on every GPU the
 * library runs on, from the loading of its code until the process ends.
 * Neither this call nor anything it enqueues allocates or frees device
 * memory; its device address is looked up (not allocated) on the first call
 * on each GPU, with that GPU made current for the lookup.
 *
 * Limits and sharing:
 *  - A call whose key splits need more than MOA_NOALLOC_SCRATCH_BYTES of
 *    partial states (moa_attn_workspace_bytes(...) with the same arguments)
 *    returns MOA_ERR_SCRATCH: decode-shaped calls, and prefill calls with
 *    num_splits > 1.  With num_splits == 0 such a prefill call runs in one
 *    pass instead, exactly as moa_attn_fwd does with too small a workspace.
 *    The automatic split choice stays within the array for every problem
 *    size whose partial states need at most 32 MiB (e.g. decode with up to
 *    B*H = 8192 heads at any Nk, or any prefill whose split items fill one
 *    wave of workgroups).
 *  - Every call on one GPU uses that GPU's one array: calls that overlap in
 *    time on the same GPU (on different streams, or from several host
 *    threads) race and may return wrong results.  Calls ordered on one stream
 *    are safe; the array keeps the last call's partial states, and nothing
 *    in it needs to start at zero.
 * Results are bit-identical to those of moa_attn_fwd with a workspace.
 */
int moa_attn_fwd_noalloc(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                         float scale, int causal, int in_dtype, int out_dtype, int num_splits,
                         void* stream);

/*
 * moa_attn_bwd_workspace_bytes -- device workspace a moa_attn_bwd call with
 * these dimensions needs, in bytes: one fp32 per query row (the row sums D
 * below), rounded up to 256 bytes.  0 for invalid or unsupported dimensions.
 */
size_t moa_attn_bwd_workspace_bytes(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk,
                                    int64_t dv);

/*
 * moa_attn_bwd -- gradients of the attention of moa_attn_fwd with respect to
 * Q, K and V (the backward pass of Sec. "Stage 5: Backward Pass and Full
 * Training Loop": dL/dQ through dL/dO, V^T, the softmax Jacobian and K, and
 * likewise for K and V).  With s_ij = scale * <q_i, k_j> over visible j:
 *
 *   P_ij  = exp(s_ij - LSE_i)            dP_ij = <dO_i, v_j>
 *   D_i   = <dO_i, O_i>                  dS_ij = P_ij * (dP_ij - D_i)
 *   dQ_i  = scale * sum_j dS_ij k_j      dK_j  = scale * sum_i dS_ij q_i
 *   dV_j  = sum_i P_ij dO_i
 *
 * The weights are recomputed from LSE: no n x n score, weight or Jacobian
 * matrix is ever written to device memory; the only writes are dQ, dK, dV
 * and the B*H*Nq row sums D in the workspace.
 *
 * Q, K, V   the forward's device inputs, bf16 (in_dtype must be MOA_BF16;
 *           MOA_F32 returns MOA_ERR_UNSUPPORTED), contiguous layouts as for
 *           moa_attn_fwd.
 * O         the forward's output, storage type o_dtype (MOA_F32 or
 *           MOA_BF16), [B][H][Nq][dv].  Only D reads it; an fp32 O gives the
 *           more accurate D.
 * dO        device input, bf16 [B][H][Nq][dv]: the gradient of the loss with
 *           respect to O.
 * LSE       the forward's LSE output, fp32 [B][H][Nq] (required).
 * dQ, dK, dV
 *           device outputs of storage type grad_dtype (MOA_F32 or MOA_BF16),
 *           shaped like Q, K, V.  Every element is written.
 * B, H, Nq, Nk, dk, dv, scale, causal
 *           exactly as passed to the forward call (same rules; dk == dv in
 *           {64, 128}).
 * workspace, workspace_bytes
 *           device scratch of at least moa_attn_bwd_workspace_bytes(...)
 *           bytes, 16-byte aligned (required when B*H*Nq > 0).
 * stream    hipStream_t as void*.
 *
 * Buffers: dQ, dK, dV and the workspace must not overlap each other or any
 * input (else MOA_ERR_INVALID_ARG); the inputs may overlap one another.  A
 * pointer may be NULL only when its tensor has no elements (Q, O, dO, LSE and
 * dQ when B*H*Nq == 0); every non-NULL pointer must be 16-byte aligned.
 * Computation: the products S, dP and the three gradient contractions run on
 * bf16 matrix cores with fp32 accumulation; P and dS are rounded to bf16
 * before they multiply dO, K and Q; exponentials and D are fp32.  Each
 * gradient row is owned by one workgroup: no atomics, and the results are
 * deterministic.  Three kernels are enqueued on `stream`.
 *
 * Returns MOA_OK once the work is enqueued (or when B*H == 0: nothing is
 * launched; when Nq == 0, dK and dV are zero-filled), else a MOA_ERR_* code.
 */
int moa_attn_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, void* dQ, void* dK, void* dV, int64_t B, int64_t H, int64_t Nq,
                 int64_t Nk, int64_t dk, int64_t dv, float scale, int causal, int in_dtype,
                 int o_dtype, int grad_dtype, void* workspace, size_t workspace_bytes,
                 void* stream);

/*
 * moa_attn_proj_workspace_bytes -- device workspace a moa_attn_fwd_proj call
 * with these dimensions needs, in bytes: the projected Q, K and V (bf16,
 * B*H*N*d elements each, every one rounded up to 256 bytes) followed by the
 * workspace moa_attn_fwd needs for the attention of those tensors.  0 for
 * invalid or unsupported dimensions.
 */
size_t moa_attn_proj_workspace_bytes(int64_t B, int64_t N, int64_t Dm, int64_t H, int64_t d);

/*
 * moa_attn_fwd_proj -- self-attention of a sequence through its input
 * projections: the paper's problem statement forms Q = X W_Q, K = X W_K,
 * V = X W_V from the sequence X and then takes Attention(Q, K, V) (Sec. "MoA
 * DNF Derivation of Attention", eq. attention), here for H heads of size d:
 *
 *   Q[b,h,n,e] = sum_k X[b,n,k] * W_Q[k, h*d + e]      (likewise K, V)
 *   O[b,h,:,:] = attention of moa_attn_fwd on Q, K, V (Nq = Nk = N)
 *
 * X         device input, bf16 [B][N][Dm] (token rows, Dm contiguous).
 * Wq, Wk, Wv
 *           device inputs, bf16 [H*d][Dm]: each weight matrix TRANSPOSED,
 *           Wq[f][k] = W_Q[k][f] (the row-major layout of a dense layer's
 *           weight; the k index is contiguous, as in X).
 * O, LSE    as for moa_attn_fwd, [B][H][N][d] (out_dtype MOA_F32 or
 *           MOA_BF16) and optional fp32 [B][H][N].
 * B, N, Dm, H, d
 *           batch, tokens per sequence, model width, heads, head size.
 *           Supported: d in {64, 128}, Dm a multiple of 64.
 * scale, causal
 *           as for moa_attn_fwd (Nq = Nk = N).
 * workspace, workspace_bytes
 *           device scratch of at least moa_attn_proj_workspace_bytes(...)
 *           bytes, 16-byte aligned (required when B*H*N > 0).  On return the
 *           projected Q, K, V sit at its start (bf16 [B][H][N][d] each, at
 *           byte offsets 0, S and 2 S with S = B*H*N*d*2 rounded up to 256).
 * stream    hipStream_t as void*.
 *
 * Computation: the three projections are one bf16 matrix-core product with
 * fp32 accumulation, rounded to bf16 (nearest even) as they are stored; the
 * attention then runs exactly as moa_attn_fwd on bf16 inputs.  Nothing but
 * Q, K, V (and the attention's own partial states when it splits its keys)
 * is written besides O and LSE.
 *
 * Buffers: O, LSE and the workspace must not overlap each other or X, Wq, Wk,
 * Wv (else MOA_ERR_INVALID_ARG).  Pointers may be NULL only when B*H*N == 0
 * (LSE: always).  Returns MOA_OK once the work is enqueued (or when
 * B*H*N == 0: nothing is launched), else a MOA_ERR_* code; an unsupported d
 * or Dm gives MOA_ERR_UNSUPPORTED.
 */
int moa_attn_fwd_proj(const void* X, const void* Wq, const void* Wk, const void* Wv, void* O,
                      float* LSE, int64_t B, int64_t N, int64_t Dm, int64_t H, int64_t d,
                      float scale, int causal, int out_dtype, void* workspace,
                      size_t workspace_bytes, void* stream);

/* moa_attn_status_string -- static, human-readable text for a status code. */
const char* moa_attn_status_string(int status);

/*
 * moa_attn_last_hip_error -- name of the HIP runtime error (e.g.
 * "hipErrorInvalidDeviceFunction") behind the most recent MOA_ERR_HIP
 * returned on the calling thread; "hipSuccess" if there was none.  Static
 * string, never NULL.
 */
const char* moa_attn_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MOA_ATTN_H */
