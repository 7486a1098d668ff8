// Internal launch interface between the C-ABI front end (api.cpp) and the
// kernels.  Not installed; the public interface is include/moa_attn.h.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace moa {

// Element strides of Q, K, V and O over batch and head (64-bit) and over
// rows (32-bit); the d dimension of every tensor is contiguous.  Contiguous
// [B][H][N][d] tensors have (batch, head, row) strides (H*N*d, N*d, d).
struct Layout {
    long long qb, qh, kb, kh, vb, vh, ob, oh;
    int qr, kr, vr, orow;
    int H;             // heads, to split a (batch*head) index
};

// One fused-attention problem after validation.  Pointers are device
// pointers; sizes are already checked to fit the kernels' 32-bit in-head
// offsets.
struct Problem {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    float* lse;        // nullable
    int bh;            // B*H
    int nq, nk, d;     // d = dk = dv
    float scale;
    bool causal;
    bool in_bf16;
    bool out_bf16;
    Layout lay;
    // Key splits of a split-K launch (1 = none) and its fp32 workspace:
    // partial states [bh * nq][splits][d] followed by [bh * nq][splits][2].
    int splits;
    float* ws;
};

// True if every tensor of `p` has the contiguous [B][H][N][d] strides.
inline bool is_contiguous(const Problem& p) {
    const Layout& L = p.lay;
    const long long d = p.d, nq = p.nq, nk = p.nk, H = L.H;
    return L.qr == d && L.qh == nq * d && L.qb == H * nq * d && L.kr == d && L.kh == nk * d &&
           L.kb == H * nk * d && L.vr == d && L.vh == nk * d && L.vb == H * nk * d &&
           L.orow == d && L.oh == nq * d && L.ob == H * nq * d;
}

// Element strides of Q, K, V and O over (batch, head, row, head element),
// any non-negative values (a column-major head has row stride 1 and element
// stride N); the tensors of the gather kernel.
struct GatherLayout {
    long long q[4], k[4], v[4], o[4];
    int H;             // heads, to split a (batch*head) index
};

// Any layout, fp32 or bf16 inputs, Nq >= 1: one launch of the element-gather
// kernel (vector ALU, fp32 arithmetic).  Uses p.q/k/v/o/lse, p.bh, p.nq,
// p.nk, p.d, p.scale, p.causal, p.in_bf16 and p.out_bf16.
hipError_t launch_prefill_gather(const Problem& p, const GatherLayout& g, hipStream_t stream);

// Prefill, bf16 inputs: one launch of the MFMA tile kernel.
hipError_t launch_prefill_bf16(const Problem& p, hipStream_t stream);


// Prefill, fp32 inputs: one launch of the fp32 vector-ALU tile kernel.
hipError_t launch_prefill_f32(const Problem& p, hipStream_t stream);

// Decode (Nq == 1): split-K partial kernel + combine kernel.
// `ws` holds bh*splits*(d + 2) floats.
hipError_t launch_decode(const Problem& p, int splits, float* ws, hipStream_t stream);

// Second pass of a split-K launch: merges the `splits` partial states of each
// of the bh * nq query rows (ws_acc [rows][splits][d], ws_ml [rows][splits][2])
// into O (and LSE when p.lse is set).
hipError_t launch_split_combine(const Problem& p, int splits, const float* ws_acc,
                                const float* ws_ml, hipStream_t stream);

// One backward problem after validation (contiguous [B][H][N][d] tensors).
// q, k, v, dout: bf16; o: bf16 or fp32; lse: fp32 natural-log LSE of the
// forward; dsum: workspace of bh*nq floats; dq, dk, dv: fp32 or bf16.
struct BwdProblem {
    const void* q;
    const void* k;
    const void* v;
    const void* o;
    const void* dout;
    const float* lse;
    float* dsum;
    void* dq;
    void* dk;
    void* dv;
    int bh;
    int nq, nk, d;
    float scale;
    bool causal;
    bool o_bf16;
    bool grad_bf16;
};

// Backward: row-dot kernel (D), dQ kernel, dK/dV kernel, in stream order.
hipError_t launch_bwd(const BwdProblem& p, hipStream_t stream);

// Bytes of the fixed device scratch array of moa_attn_fwd_noalloc (one per
// GPU, held until the process ends; equal to MOA_NOALLOC_SCRATCH_BYTES).
constexpr size_t kNoallocScratchBytes = size_t(32) << 20;

// Device address of the scratch array on the GPU that runs `stream`, looked up
// once per device (with that device current) and cached; allocates nothing.
hipError_t noalloc_scratch(hipStream_t stream, void** ptr);

// Row-tile size of the bf16 prefill kernel (queries per workgroup).
constexpr int kPrefillBf16RowsPerBlock = 256;
// Row-tile size of the fp32 prefill kernel.
constexpr int kPrefillF32RowsPerBlock = 16;
// Row-tile size of the element-gather kernel.
constexpr int kPrefillGatherRowsPerBlock = 64;

}  // namespace moa
