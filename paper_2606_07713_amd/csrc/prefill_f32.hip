// Fused attention prefill for fp32 inputs and fp32 output (vector ALU, fp32
// throughout).
//
// Used where the inputs are fp32 and the result must stay within fp32
// rounding of the exact attention (no bf16 rounding of any operand).  One
// workgroup owns a tile of query rows of one (batch*head); each row is
// handled by QL lanes that split d (4, 8 or 16).  The waves of a workgroup hold
// the same rows and walk disjoint key streams (wave w takes tiles w,
// w + STREAMS, ...; 128 keys per round of the workgroup), each staging its
// own K/V tiles in its own LDS area, read by its lanes as broadcasts.  At the
// end every wave stores its softmax state and all threads merge the streams
// exactly, one float4 of O each.  The key split keeps each wave's chain of
// dependent loads and vector instructions short, which is what these small
// problems are bound by.  Scores, the running max and sum and the
// exponentials stay in registers (DNF eqs. dnf_attn / output_dnf); only O
// (and optional LSE) are written.
#include "device_common.h"
#include "launch.h"
#include "prefill_bf16_common.h"   // device_cus

namespace moa {
namespace {

constexpr int ROUND_KEYS = 128;   // keys per round of all streams (STREAMS x KT)

// QL lanes share a query row (they split d); a wave holds 64 / QL rows, and
// every wave of a workgroup holds the same rows.
template <int QL>
constexpr int rows_of() { return 64 / QL; }
template <int STREAMS>
constexpr int threads_of() { return 64 * STREAMS; }

template <int D, bool CAUSAL, int STREAMS, int QL>
__global__ __launch_bounds__(threads_of<STREAMS>()) void prefill_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    float* __restrict__ Out, float* __restrict__ LSE, int Nq, int Nk, int n_qtiles, float c,
    Layout L) {
    constexpr int THREADS = threads_of<STREAMS>();
    constexpr int ROWS = rows_of<QL>();
    constexpr int KT = ROUND_KEYS / STREAMS;   // keys per tile
    constexpr int CH = D / (4 * QL);   // float4 chunks per lane (chunk j*QL + quad)
    constexpr int TILE = KT * D;  // floats of one K (or V) tile
    constexpr int PER = TILE / 4 / 64;   // float4 per lane per tile
    static_assert(TILE % 256 == 0, "a tile must split into whole float4 per lane");
    // Per wave: its K tile followed by its V tile.  After the key loop the
    // same area holds the wave's un-normalised output, ROWS x D floats.
    static_assert(ROWS * D <= 2 * TILE, "a wave's K and V tiles must hold its output rows");
    __shared__ __attribute__((aligned(16))) float KV[STREAMS][2 * TILE];
    __shared__ float ML[STREAMS][2][ROWS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // key stream
    const int quad = lane % QL;   // this lane's part of the row
    const int row = lane / QL;
    const int bh = blockIdx.x / n_qtiles;
    const int qt = blockIdx.x % n_qtiles;
    const int qrow = qt * ROWS + row;
    const int qrow_c = qrow < Nq ? qrow : Nq - 1;
    const int off = Nk - Nq;

    const float* Qh = Q + head_offset(bh, L.H, L.qb, L.qh);
    const float* Kh = K + head_offset(bh, L.H, L.kb, L.kh);
    const float* Vh = V + head_offset(bh, L.H, L.vb, L.vh);
    float* ks = KV[wave];
    float* vs = KV[wave] + TILE;

    float4 qv[CH], acc[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        qv[j] = *reinterpret_cast<const float4*>(Qh + (size_t)qrow_c * L.qr + (j * QL + quad) * 4);
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
        float4 kst[PER], vst[PER];
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = i * 64 + lane;
            const int r = idx / (D / 4), ch = idx % (D / 4);
            const int key = min(kbase + r, Nk - 1);
            kst[i] = *reinterpret_cast<const float4*>(Kh + (size_t)key * L.kr + ch * 4);
            vst[i] = *reinterpret_cast<const float4*>(Vh + (size_t)key * L.vr + ch * 4);
        }
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = i * 64 + lane;
            const int r = idx / (D / 4), ch = idx % (D / 4);
            *reinterpret_cast<float4*>(&ks[r * D + ch * 4]) = kst[i];
            *reinterpret_cast<float4*>(&vs[r * D + ch * 4]) = vst[i];
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
                const float4 kk = *reinterpret_cast<const float4*>(&ks[j * D + (h * QL + quad) * 4]);
                part = __builtin_fmaf(qv[h].x, kk.x, part);
                part = __builtin_fmaf(qv[h].y, kk.y, part);
                part = __builtin_fmaf(qv[h].z, kk.z, part);
                part = __builtin_fmaf(qv[h].w, kk.w, part);
            }
            const float s = group_sum<QL>(part);
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
                const float4 vv = *reinterpret_cast<const float4*>(&vs[j * D + (h * QL + quad) * 4]);
                acc[h].x = __builtin_fmaf(p, vv.x, acc[h].x);
                acc[h].y = __builtin_fmaf(p, vv.y, acc[h].y);
                acc[h].z = __builtin_fmaf(p, vv.z, acc[h].z);
                acc[h].w = __builtin_fmaf(p, vv.w, acc[h].w);
            }
        }
    }

    // Exact merge of the streams' states: every wave stores (m, l, acc) of
    // its stream, then each thread finishes one float4 of O:
    //   M = max_w m_w,  O = sum_w 2^(m_w - M) acc_w / sum_w 2^(m_w - M) l_w.
    // A stream without visible keys has m = -inf and adds nothing.
    __syncthreads();   // every wave is done reading its tiles
#pragma unroll
    for (int h = 0; h < CH; ++h)
        *reinterpret_cast<float4*>(&ks[row * D + (h * QL + quad) * 4]) = acc[h];
    if (quad == 0) {
        ML[wave][0][row] = m_run;
        ML[wave][1][row] = l_run;
    }
    __syncthreads();
    constexpr int OUT4 = ROWS * D / 4;   // float4 of the workgroup's output
    for (int t = threadIdx.x; t < OUT4; t += THREADS) {
        const int r = t / (D / 4), c4 = t % (D / 4);
        float mm = kNegInf;
#pragma unroll
        for (int w = 0; w < STREAMS; ++w) mm = fmaxf(mm, ML[w][0][r]);
        float ll = 0.0f;
        float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int w = 0; w < STREAMS; ++w) {
            const float mw = ML[w][0][r];
            const float a = (mw == kNegInf) ? 0.0f : exp2_hw(mw - mm);
            ll = __builtin_fmaf(a, ML[w][1][r], ll);
            const float4 x = *reinterpret_cast<const float4*>(&KV[w][r * D + c4 * 4]);
            o.x = __builtin_fmaf(a, x.x, o.x);
            o.y = __builtin_fmaf(a, x.y, o.y);
            o.z = __builtin_fmaf(a, x.z, o.z);
            o.w = __builtin_fmaf(a, x.w, o.w);
        }
        const int q = qt * ROWS + r;
        if (q < Nq) {
            const float inv = 1.0f / ll;
            const size_t obase = (size_t)head_offset(bh, L.H, L.ob, L.oh) + (size_t)q * L.orow;
            *reinterpret_cast<float4*>(Out + obase + c4 * 4) =
                make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv);
            if (LSE != nullptr && c4 == 0) LSE[(size_t)bh * Nq + q] = (mm + __log2f(ll)) * kLn2;
        }
    }
}

// Four shapes of workgroup, by grid size (raw C-ABI calls, us, one box):
//
//   streams x key tile, lanes per row, rows   8x16,4,16  16x8,4,16  16x8,8,8  16x8,16,4
//   B1 H1 128 x 128, d = 64                    6.39       6.83       4.97      4.57
//   B1 H1 128 x 128, d = 128                   9.73       10.27      6.73      5.40
//   B1 H2 300 x 517, d = 128                   31.7       27.9       17.1      13.3
//   B1 H1 1K x 1K causal, d = 64               -          -          17.2      14.5
//   B1 H1 2K x 2K causal, d = 128              103.1      88.9       56.5      56.4
//   B1 H1 4K x 4K, d = 64                      128.8      121.4      146.6     -
//   B4 H8 256 x 256, d = 64                    16.5       17.7       22.4      -
//   B1 H16 1K x 1K, d = 64                     100.9      101.2      140.7     -
//
// Splitting a row over more lanes shortens each wave's chain and multiplies
// the grid; it pays while the grid still fits the GPU.  So: 16 lanes per row
// (4 rows per workgroup) while that grid fits the compute units, else 8 lanes
// (8 rows) while that one does, all with sixteen key streams; long keys on
// grids of up to one 16-row workgroup per unit take sixteen streams of 16
// rows; everything else eight streams of 16 rows, whose workgroups are the
// cheapest to start and merge.
constexpr int kWideMinKeys = 512;

template <int D, bool CAUSAL, int STREAMS, int QL>
hipError_t launch_s(const Problem& p, hipStream_t stream) {
    constexpr int ROWS = rows_of<QL>();
    const int n_qtiles = (p.nq + ROWS - 1) / ROWS;
    const long long blocks = (long long)p.bh * n_qtiles;
    return launch_kernel(prefill_f32_kernel<D, CAUSAL, STREAMS, QL>, dim3((unsigned)blocks),
                         dim3(threads_of<STREAMS>()), stream, static_cast<const float*>(p.q),
                         static_cast<const float*>(p.k), static_cast<const float*>(p.v),
                         static_cast<float*>(p.o), p.lse, p.nq, p.nk, n_qtiles,
                         p.scale * kLog2e, p.lay);
}

template <int D, bool CAUSAL>
hipError_t launch(const Problem& p, hipStream_t stream) {
    const long long blocks16 = (long long)p.bh * ((p.nq + 15) / 16);
    int cus = 0;
    const hipError_t e = pf::device_cus(stream, cus);
    if (e != hipSuccess) return e;
    if (4 * blocks16 <= cus) return launch_s<D, CAUSAL, 16, 16>(p, stream);
    if (2 * blocks16 <= cus) return launch_s<D, CAUSAL, 16, 8>(p, stream);
    if (p.nk >= kWideMinKeys && blocks16 <= cus) return launch_s<D, CAUSAL, 16, 4>(p, stream);
    return launch_s<D, CAUSAL, 8, 4>(p, stream);
}

template <int D>
hipError_t launch_d(const Problem& p, hipStream_t stream) {
    return p.causal ? launch<D, true>(p, stream) : launch<D, false>(p, stream);
}

}  // namespace

static_assert(rows_of<4>() == kPrefillF32RowsPerBlock, "row tile mismatch");

hipError_t launch_prefill_f32(const Problem& p, hipStream_t stream) {
    if (p.d == 64) return launch_d<64>(p, stream);
    if (p.d == 128) return launch_d<128>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
