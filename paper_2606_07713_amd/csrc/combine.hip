// Exact merge of per-split partial softmax states (the second pass of every
// split-K launch: decode, and prefill on grids too small to fill the GPU).
//
// A split s of query row r holds, over its own key range only, the reference
// m_s (log2 units, s_j * scale * log2(e)), the denominator l_s = sum_j
// 2^(s_j - m_s) and the un-normalised output acc_s = sum_j 2^(s_j - m_s) v_j.
// With M = max_s m_s,
//   O_r = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s,
// which is the DNF's denominator sum (eq. dnf_attn) and the contraction of
// eq. output_dnf regrouped over key ranges: exact in exact arithmetic.  Splits
// that saw no visible key (m_s = -inf, l_s = 0) contribute nothing.
#include "device_common.h"
#include "launch.h"

namespace moa {
namespace {

constexpr int ROWS_PER_BLOCK = 4;   // one wave per query row

// ws_acc: [rows][splits][D] fp32, ws_ml: [rows][splits][2] fp32 (m, l), with
// row = bh * nq + i.  O is written through the layout's strides.
template <int D, bool OUT_BF16>
__global__ __launch_bounds__(ROWS_PER_BLOCK * 64) void split_combine_kernel(
    const float* __restrict__ ws_acc, const float* __restrict__ ws_ml, void* __restrict__ Out,
    float* __restrict__ LSE, long long rows, int nq, int splits, Layout lay) {
    constexpr int PER = D / 64;
    const long long row = (long long)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const float* ml = ws_ml + (size_t)row * splits * 2;
    const float* ac = ws_acc + (size_t)row * splits * D;
    float M = kNegInf;
    for (int s = 0; s < splits; ++s) M = fmaxf(M, ml[2 * s]);
    float L = 0.0f, o[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] = 0.0f;
    for (int s = 0; s < splits; ++s) {
        const float ms = ml[2 * s];
        const float w = (ms == kNegInf) ? 0.0f : exp2_hw(ms - M);
        L += w * ml[2 * s + 1];
#pragma unroll
        for (int e = 0; e < PER; ++e) o[e] += w * ac[(size_t)s * D + e * 64 + lane];
    }
    const float inv = 1.0f / L;
    const int bh = (int)(row / nq);
    const int i = (int)(row - (long long)bh * nq);
    const size_t base = (size_t)head_offset(bh, lay.H, lay.ob, lay.oh) + (size_t)i * lay.orow;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        if (OUT_BF16)
            static_cast<u16*>(Out)[base + e * 64 + lane] = (u16)f32_to_bf16_bits(o[e] * inv);
        else
            static_cast<float*>(Out)[base + e * 64 + lane] = o[e] * inv;
    }
    if (LSE != nullptr && lane == 0) LSE[row] = (M + __log2f(L)) * kLn2;
}

template <int D>
hipError_t launch_d(const Problem& p, int splits, const float* ws_acc, const float* ws_ml,
                    hipStream_t stream) {
    const long long rows = (long long)p.bh * p.nq;
    const unsigned grid = (unsigned)((rows + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK);
    if (p.out_bf16)
        return launch_kernel(split_combine_kernel<D, true>, dim3(grid), dim3(ROWS_PER_BLOCK * 64),
                             stream, ws_acc, ws_ml, p.o, p.lse, rows, p.nq, splits, p.lay);
    return launch_kernel(split_combine_kernel<D, false>, dim3(grid), dim3(ROWS_PER_BLOCK * 64),
                         stream, ws_acc, ws_ml, p.o, p.lse, rows, p.nq, splits, p.lay);
}

}  // namespace

hipError_t launch_split_combine(const Problem& p, int splits, const float* ws_acc,
                                const float* ws_ml, hipStream_t stream) {
    if (p.bh == 0 || p.nq == 0) return hipSuccess;
    if (p.d == 64) return launch_d<64>(p, splits, ws_acc, ws_ml, stream);
    if (p.d == 128) return launch_d<128>(p, splits, ws_acc, ws_ml, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
