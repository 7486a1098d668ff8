// Decode-shaped attention (one query per (batch, head)): split-K + combine.
//
// The work is pure streaming of K and V (one multiply-add per loaded element),
// so it is bound by device-memory bandwidth.  The key range of each
// (batch*head) is cut into `splits` chunks; one workgroup streams one chunk
// with coalesced 16-byte loads, many loads in flight per lane, and reduces it
// to a partial softmax state (m_s, l_s, acc_s[dv]) in fp32 -- the row max of
// Step I, the denominator of Step III and the un-normalised output of eq.
// output_dnf, all restricted to the chunk's keys.  A second kernel merges the
// partial states exactly:  M = max_s m_s,
//   O = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s,
// which is the DNF's denominator sum (eq. dnf_attn) regrouped over key chunks.
// Only the partial states (O(B*H*splits*dv)) and O itself are written.
#include "device_common.h"
#include "launch.h"

namespace moa {
namespace {

constexpr int WAVES = 4;
constexpr int THREADS = WAVES * 64;
constexpr int U = 8;   // 16-byte K (and V) loads per lane in flight per iteration

template <typename T, int D>
struct Cfg {
    static constexpr int EPL = 16 / (int)sizeof(T);   // elements per 16-byte load
    static constexpr int LPR = D / EPL;               // lanes per key row
    static constexpr int RPW = 64 / LPR;              // key rows per wave per load
    static constexpr int STEP = RPW * U;              // keys per wave per iteration
    static_assert(LPR >= 1 && LPR <= 64 && 64 % LPR == 0, "bad row split");
};

template <typename T>
__device__ __forceinline__ void widen(const uint4& w, float (&x)[16 / sizeof(T)]);

template <>
__device__ __forceinline__ void widen<u16>(const uint4& w, float (&x)[8]) {
    x[0] = bf16lo_to_f32(w.x); x[1] = bf16hi_to_f32(w.x);
    x[2] = bf16lo_to_f32(w.y); x[3] = bf16hi_to_f32(w.y);
    x[4] = bf16lo_to_f32(w.z); x[5] = bf16hi_to_f32(w.z);
    x[6] = bf16lo_to_f32(w.w); x[7] = bf16hi_to_f32(w.w);
}

template <>
__device__ __forceinline__ void widen<float>(const uint4& w, float (&x)[4]) {
    x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
    x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
}

// Merge the softmax state (m, l, acc) with the one held `OFF` lanes away.
template <int EPL, int OFF>
__device__ __forceinline__ void merge_xor(float& m, float& l, float (&acc)[EPL]) {
    const float m2 = __shfl_xor(m, OFF);
    const float l2 = __shfl_xor(l, OFF);
    const float mm = fmaxf(m, m2);
    const float a1 = (m == kNegInf) ? 0.0f : exp2_hw(m - mm);
    const float a2 = (m2 == kNegInf) ? 0.0f : exp2_hw(m2 - mm);
    l = l * a1 + l2 * a2;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
        const float o2 = __shfl_xor(acc[e], OFF);
        acc[e] = acc[e] * a1 + o2 * a2;
    }
    m = mm;
}

// a8: one workgroup = one key chunk of one (batch*head).  DIRECT (one chunk
// per row): the workgroup holds the row's whole softmax state, so it writes
// O = acc / l (and LSE) itself -- the value the combine pass would compute
// from a single split, where every merge weight is exactly 1 -- instead of
// the partial state, and no combine pass runs.
template <typename T, int D, bool DIRECT = false, bool OUT_BF16 = false>
__global__ __launch_bounds__(THREADS) void decode_split_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    float* __restrict__ ws_acc, float* __restrict__ ws_ml, int Nk, int splits,
    int keys_per_split, float c, Layout L, void* __restrict__ Out, float* __restrict__ LSE) {
    using C = Cfg<T, D>;
    constexpr int EPL = C::EPL, LPR = C::LPR, RPW = C::RPW, STEP = C::STEP;
    __shared__ float red_m[WAVES], red_l[WAVES];
    __shared__ __attribute__((aligned(16))) float red_acc[WAVES][D];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = lane / LPR;   // key row within a load
    const int el = lane % LPR;    // which EPL-element chunk of the row
    const int bh = blockIdx.x / splits;
    const int sp = blockIdx.x % splits;
    const int k_begin = sp * keys_per_split;
    const int k_end = min(Nk, k_begin + keys_per_split);

    const T* Kh = K + head_offset(bh, L.H, L.kb, L.kh);
    const T* Vh = V + head_offset(bh, L.H, L.vb, L.vh);
    float qv[EPL];
    widen<T>(*reinterpret_cast<const uint4*>(Q + head_offset(bh, L.H, L.qb, L.qh) + el * EPL), qv);

    float m = kNegInf, l = 0.0f, acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.0f;

    for (int kb = k_begin + wave * STEP; kb < k_end; kb += WAVES * STEP) {
        uint4 kr[U], vr[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int key = min(kb + u * RPW + grp, k_end - 1);
            kr[u] = load_nt16(Kh + (size_t)key * L.kr + el * EPL);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int key = min(kb + u * RPW + grp, k_end - 1);
            vr[u] = load_nt16(Vh + (size_t)key * L.vr + el * EPL);
        }
        // scores (log2 units) of the U keys this lane group holds
        float t[U];
        float tmax = kNegInf;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float kx[EPL];
            widen<T>(kr[u], kx);
            float part = 0.0f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) part = __builtin_fmaf(qv[e], kx[e], part);
            const float s = group_sum<LPR>(part);
            t[u] = (kb + u * RPW + grp < k_end) ? s * c : kNegInf;
            tmax = fmaxf(tmax, t[u]);
        }
        const float m_new = fmaxf(m, tmax);
        if (m_new != kNegInf) {
            const float alpha = (m == kNegInf) ? 0.0f : exp2_hw(m - m_new);
            l *= alpha;
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[e] *= alpha;
            m = m_new;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float p = (t[u] == kNegInf) ? 0.0f : exp2_hw(t[u] - m);
            l += p;
            float vx[EPL];
            widen<T>(vr[u], vx);
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[e] = __builtin_fmaf(p, vx[e], acc[e]);
        }
    }

    // Merge the RPW lane groups of the wave, then the waves through LDS.
    if constexpr (RPW >= 2) merge_xor<EPL, LPR * 1>(m, l, acc);
    if constexpr (RPW >= 4) merge_xor<EPL, LPR * 2>(m, l, acc);
    if constexpr (RPW >= 8) merge_xor<EPL, LPR * 4>(m, l, acc);
    if constexpr (RPW >= 16) merge_xor<EPL, LPR * 8>(m, l, acc);
    if (lane < LPR) {
        if (lane == 0) { red_m[wave] = m; red_l[wave] = l; }
#pragma unroll
        for (int e = 0; e < EPL; ++e) red_acc[wave][el * EPL + e] = acc[e];
    }
    __syncthreads();
    if (wave == 0 && lane < LPR) {
        float mm = kNegInf;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) mm = fmaxf(mm, red_m[w]);
        float ll = 0.0f, o[EPL];
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[e] = 0.0f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            const float a = (red_m[w] == kNegInf) ? 0.0f : exp2_hw(red_m[w] - mm);
            ll += a * red_l[w];
#pragma unroll
            for (int e = 0; e < EPL; ++e) o[e] += a * red_acc[w][el * EPL + e];
        }
        if constexpr (DIRECT) {
            const float inv = 1.0f / ll;
            const size_t base = (size_t)head_offset(bh, L.H, L.ob, L.oh) + (size_t)el * EPL;
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
                if constexpr (OUT_BF16)
                    static_cast<u16*>(Out)[base + e] = (u16)f32_to_bf16_bits(o[e] * inv);
                else
                    static_cast<float*>(Out)[base + e] = o[e] * inv;
            }
            if (LSE != nullptr && lane == 0) LSE[bh] = (mm + __log2f(ll)) * kLn2;
        } else {
            const size_t row = (size_t)bh * splits + sp;
#pragma unroll
            for (int e = 0; e < EPL; ++e) ws_acc[row * D + el * EPL + e] = o[e];
            if (lane == 0) {
                ws_ml[row * 2 + 0] = mm;
                ws_ml[row * 2 + 1] = ll;
            }
        }
    }
}

template <typename T, int D>
hipError_t launch_t(const Problem& p, int splits, float* ws, hipStream_t stream) {
    const int kps = (p.nk + splits - 1) / splits;
    float* ws_acc = ws;
    float* ws_ml = ws + (size_t)p.bh * splits * D;
    const long long blocks = (long long)p.bh * splits;
    const auto args = [&](auto kernel) {
        return launch_kernel(kernel, dim3((unsigned)blocks), dim3(THREADS), stream,
                             static_cast<const T*>(p.q), static_cast<const T*>(p.k),
                             static_cast<const T*>(p.v), ws_acc, ws_ml, p.nk, splits, kps,
                             p.scale * kLog2e, p.lay, p.o, p.lse);
    };
    if (splits == 1)
        return p.out_bf16 ? args(decode_split_kernel<T, D, true, true>)
                          : args(decode_split_kernel<T, D, true, false>);
    const hipError_t e = args(decode_split_kernel<T, D>);
    if (e != hipSuccess) return e;
    // a9: exact merge of the per-chunk states (one query row per batch*head).
    return launch_split_combine(p, splits, ws_acc, ws_ml, stream);
}

}  // namespace

hipError_t launch_decode(const Problem& p, int splits, float* ws, hipStream_t stream) {
    if (p.in_bf16) {
        if (p.d == 64) return launch_t<u16, 64>(p, splits, ws, stream);
        if (p.d == 128) return launch_t<u16, 128>(p, splits, ws, stream);
    } else {
        if (p.d == 64) return launch_t<float, 64>(p, splits, ws, stream);
        if (p.d == 128) return launch_t<float, 128>(p, splits, ws, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace moa
