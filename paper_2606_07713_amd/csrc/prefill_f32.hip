// Fused attention prefill for fp32 inputs and fp32 output (vector ALU, fp32
// throughout).
//
// Used where the inputs are fp32 and the result must stay within fp32
// rounding of the exact attention (no bf16 rounding of any operand).  One
// workgroup owns 16 queries of one (batch*head); each query row is handled by
// a quad of 4 lanes that split d.  The eight waves of a workgroup hold the
// same queries and walk disjoint key streams (wave w takes 16-key tiles w,
// w + 8, ...), each staging its own K/V tiles in its own LDS area, read by its
// quads as broadcasts; at the end waves 1..7 hand their softmax state to wave
// 0, which merges it exactly.  The key split keeps each wave's chain of
// dependent loads and vector instructions short, which is what these small
// problems are bound by (8 streams of 16 keys measured 24-40% faster than 4
// streams of 32 keys, on 128 x 128 single heads up to 1K causal grids).  Scores, the
// running max and sum and the exponentials stay in registers (DNF eqs.
// dnf_attn / output_dnf); only O (and optional LSE) are written.
#include "device_common.h"
#include "launch.h"

namespace moa {
namespace {

constexpr int ROWS = 16;          // queries per workgroup
constexpr int STREAMS = 8;        // key streams (waves) per workgroup
constexpr int THREADS = ROWS * 4 * STREAMS;
constexpr int KT = 16;            // keys per tile

template <int D, bool CAUSAL>
__global__ __launch_bounds__(THREADS) void prefill_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    float* __restrict__ Out, float* __restrict__ LSE, int Nq, int Nk, int n_qtiles, float c,
    Layout L) {
    constexpr int CH = D / 16;    // float4 chunks per lane (chunk j*4 + quad)
    // Per wave: its K and V tile; reused at the end for the merge, where a K
    // tile holds the wave's O (D / 4 floats per lane: KT >= 16 keys).
    static_assert(KT * D >= 64 * (D / 4), "a K tile must hold one wave's O for the merge");
    __shared__ __attribute__((aligned(16))) float Ks[STREAMS][KT * D];
    __shared__ __attribute__((aligned(16))) float Vs[STREAMS][KT * D];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // key stream
    const int quad = lane & 3;
    const int bh = blockIdx.x / n_qtiles;
    const int qt = blockIdx.x % n_qtiles;
    const int qrow = qt * ROWS + (lane >> 2);
    const int qrow_c = qrow < Nq ? qrow : Nq - 1;
    const int off = Nk - Nq;

    const float* Qh = Q + head_offset(bh, L.H, L.qb, L.qh);
    const float* Kh = K + head_offset(bh, L.H, L.kb, L.kh);
    const float* Vh = V + head_offset(bh, L.H, L.vb, L.vh);
    float* ks = Ks[wave];
    float* vs = Vs[wave];

    float4 qv[CH], acc[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        qv[j] = *reinterpret_cast<const float4*>(Qh + (size_t)qrow_c * L.qr + (j * 4 + quad) * 4);
        acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float m_run = kNegInf, l_run = 0.0f;

    int kv_end = Nk;
    if (CAUSAL) kv_end = min(Nk, qt * ROWS + ROWS + off);
    const int n_kt = (kv_end + KT - 1) / KT;

    for (int kt = wave; kt < n_kt; kt += STREAMS) {
        const int kbase = kt * KT;
        // This wave's tile: its own LDS area, so only its own accesses need
        // ordering (every lane's previous reads are consumed, its stores land
        // before the reads below).
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        constexpr int PER = KT * D / 4 / 64;  // float4 per lane per tile
        float4 kst[PER], vst[PER];
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = i * 64 + lane;
            const int row = idx / (D / 4), ch = idx % (D / 4);
            const int key = min(kbase + row, Nk - 1);
            kst[i] = *reinterpret_cast<const float4*>(Kh + (size_t)key * L.kr + ch * 4);
            vst[i] = *reinterpret_cast<const float4*>(Vh + (size_t)key * L.vr + ch * 4);
        }
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = i * 64 + lane;
            const int row = idx / (D / 4), ch = idx % (D / 4);
            *reinterpret_cast<float4*>(&ks[row * D + ch * 4]) = kst[i];
            *reinterpret_cast<float4*>(&vs[row * D + ch * 4]) = vst[i];
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the stores have landed
        __builtin_amdgcn_wave_barrier();

        // scores of this tile, in log2 units (t = c * <q, k>)
        float t[KT];
        float tmax = kNegInf;
#pragma unroll
        for (int j = 0; j < KT; ++j) {
            float part = 0.0f;
#pragma unroll
            for (int h = 0; h < CH; ++h) {
                const float4 kk = *reinterpret_cast<const float4*>(&ks[j * D + (h * 4 + quad) * 4]);
                part = __builtin_fmaf(qv[h].x, kk.x, part);
                part = __builtin_fmaf(qv[h].y, kk.y, part);
                part = __builtin_fmaf(qv[h].z, kk.z, part);
                part = __builtin_fmaf(qv[h].w, kk.w, part);
            }
            const float s = group_sum<4>(part);
            const int key = kbase + j;
            const bool vis = key < Nk && (!CAUSAL || key <= qrow + off);
            t[j] = vis ? s * c : kNegInf;
            tmax = fmaxf(tmax, t[j]);
        }
        const float m_new = fmaxf(m_run, tmax);
        if (m_new != kNegInf) {
            const float alpha = (m_run == kNegInf) ? 0.0f : exp2_hw(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int h = 0; h < CH; ++h) {
                acc[h].x *= alpha; acc[h].y *= alpha; acc[h].z *= alpha; acc[h].w *= alpha;
            }
            m_run = m_new;
        }
#pragma unroll
        for (int j = 0; j < KT; ++j) {
            const float p = (t[j] == kNegInf) ? 0.0f : exp2_hw(t[j] - m_run);
            l_run += p;
#pragma unroll
            for (int h = 0; h < CH; ++h) {
                const float4 vv = *reinterpret_cast<const float4*>(&vs[j * D + (h * 4 + quad) * 4]);
                acc[h].x = __builtin_fmaf(p, vv.x, acc[h].x);
                acc[h].y = __builtin_fmaf(p, vv.y, acc[h].y);
                acc[h].z = __builtin_fmaf(p, vv.z, acc[h].z);
                acc[h].w = __builtin_fmaf(p, vv.w, acc[h].w);
            }
        }
    }

    // Waves 1..7 hand (m, l, acc) to wave 0 through their K areas; wave 0
    // merges exactly: M = max(m0, mw), acc = 2^(m0-M) acc0 + 2^(mw-M) accw,
    // l likewise.  A stream without visible keys has m = -inf and adds nothing.
    __syncthreads();
    if (wave != 0) {
#pragma unroll
        for (int h = 0; h < CH; ++h)
            *reinterpret_cast<float4*>(&ks[(h * 64 + lane) * 4]) = acc[h];
        vs[lane] = m_run;
        vs[64 + lane] = l_run;
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int w = 1; w < STREAMS; ++w) {
        const float m1 = Vs[w][lane], l1 = Vs[w][64 + lane];
        const float mm = fmaxf(m_run, m1);
        const float a0 = (m_run == kNegInf) ? 0.0f : exp2_hw(m_run - mm);
        const float a1 = (m1 == kNegInf) ? 0.0f : exp2_hw(m1 - mm);
        l_run = l_run * a0 + l1 * a1;
#pragma unroll
        for (int h = 0; h < CH; ++h) {
            const float4 o = *reinterpret_cast<const float4*>(&Ks[w][(h * 64 + lane) * 4]);
            acc[h].x = acc[h].x * a0 + o.x * a1;
            acc[h].y = acc[h].y * a0 + o.y * a1;
            acc[h].z = acc[h].z * a0 + o.z * a1;
            acc[h].w = acc[h].w * a0 + o.w * a1;
        }
        m_run = mm;
    }

    if (qrow < Nq) {
        const float inv = 1.0f / l_run;
        const size_t obase = (size_t)head_offset(bh, L.H, L.ob, L.oh) + (size_t)qrow * L.orow;
#pragma unroll
        for (int h = 0; h < CH; ++h) {
            const int d0 = (h * 4 + quad) * 4;
            const float4 o = make_float4(acc[h].x * inv, acc[h].y * inv, acc[h].z * inv, acc[h].w * inv);
            *reinterpret_cast<float4*>(Out + obase + d0) = o;
        }
        if (LSE != nullptr && quad == 0)
            LSE[(size_t)bh * Nq + qrow] = (m_run + __log2f(l_run)) * kLn2;
    }
}

template <int D, bool CAUSAL>
hipError_t launch(const Problem& p, hipStream_t stream) {
    const int n_qtiles = (p.nq + ROWS - 1) / ROWS;
    const long long blocks = (long long)p.bh * n_qtiles;
    return launch_kernel(prefill_f32_kernel<D, CAUSAL>, dim3((unsigned)blocks), dim3(THREADS),
                         stream, static_cast<const float*>(p.q), static_cast<const float*>(p.k),
                         static_cast<const float*>(p.v), static_cast<float*>(p.o), p.lse, p.nq,
                         p.nk, n_qtiles, p.scale * kLog2e, p.lay);
}

template <int D>
hipError_t launch_d(const Problem& p, hipStream_t stream) {
    return p.causal ? launch<D, true>(p, stream) : launch<D, false>(p, stream);
}

}  // namespace

static_assert(ROWS == kPrefillF32RowsPerBlock, "row tile mismatch");

hipError_t launch_prefill_f32(const Problem& p, hipStream_t stream) {
    if (p.d == 64) return launch_d<64>(p, stream);
    if (p.d == 128) return launch_d<128>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
