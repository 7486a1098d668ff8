// Fused attention prefill for bf16 inputs on gfx950 matrix cores.
//
// One workgroup owns one (batch*head, 128-query tile).  It keeps its Q tile in
// registers for the whole key loop, streams K and V through LDS one 64-key
// tile at a time, and never writes anything but the output (and optional LSE)
// to device memory: the score tile, the exponentials and the running softmax
// statistics live in registers only (the DNF of eqs. dnf_attn / output_dnf).
//
// Orientation.  Each wave computes the transposed score tile S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16: K rows are the A operand read straight from LDS in
// their stored order, so no K^T is ever formed (eq. mm_psi reads K by row).
// In the accumulator layout every lane then holds scores of ONE query
// (column = lane % 32) for 16 of the tile's keys, and lane l ^ 32 holds the
// other keys of the same query, so the row max (Step I) and row sum (Step III)
// are in-lane reductions plus one exchange between the two half-waves.
// The output is accumulated transposed too, O^T += V^T P^T: the P^T operand
// is the score accumulator re-packed to bf16 in place (no data movement), and
// V^T comes from an LDS copy of the V tile stored dv-major.
//
// Softmax.  Scores are kept in raw units; with c = scale * log2(e) the weight
// of key j is 2^(s_j c - m) where m is a running row maximum in log2 units.
// The running maximum is only raised (and O, l rescaled) when the tile max
// exceeds it by more than kRescaleSlack; otherwise weights up to
// 2^kRescaleSlack are accumulated against the stale maximum.  The final
// O = acc / l uses the same maximum for numerator and denominator, so the
// result is the same softmax (Steps I-IV regrouped over key tiles).
#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace moa {
namespace {

constexpr int BM = 128;          // queries per workgroup
constexpr int BN = 64;           // keys per tile
constexpr int WAVES = 4;         // each wave: 32 queries
constexpr int THREADS = WAVES * 64;
constexpr float kRescaleSlack = 8.0f;

template <int D>
struct Tile {
    static constexpr int KSTRIDE = D + 8;    // K tile row stride (elements): rows shift 4 banks
    static constexpr int VSTRIDE = BN + 4;   // V^T row stride (elements)
    static constexpr int K_ELEMS = BN * KSTRIDE;
    static constexpr int V_ELEMS = D * VSTRIDE;
    static constexpr int K_CHUNKS = BN * D / 8;             // 16-byte chunks per K tile
    static constexpr int K_PASSES = K_CHUNKS / THREADS;     // 16-byte loads per thread
    static constexpr int V_THREADS = (D / 8) * (BN / 4);    // threads loading 4 keys x 8 dv
    static_assert(K_CHUNKS % THREADS == 0, "K tile must split evenly");
    static_assert(V_THREADS <= THREADS, "V tile too large");
};

// Workgroup index -> (head slice, query tile), keeping the query tiles of one
// head on one XCD (workgroups are handed to the 8 XCDs round-robin) so that
// the K/V tiles they all stream are shared in that XCD's L2.  Within a head
// the heaviest causal tiles start first.
__device__ __forceinline__ void tile_of_block(int bid, int nblocks, int n_qtiles, bool causal,
                                              int& bh, int& qt) {
    const int per = nblocks >> 3, rem = nblocks & 7;
    const int x = bid & 7, r = bid >> 3;
    const int logical = x * per + (x < rem ? x : rem) + r;
    bh = logical / n_qtiles;
    const int t = logical - bh * n_qtiles;
    qt = causal ? (n_qtiles - 1 - t) : t;
}

template <int D, bool CAUSAL, bool OUT_BF16>
__global__ __launch_bounds__(THREADS, 2) void prefill_bf16_kernel(
    const u16* __restrict__ Q, const u16* __restrict__ K, const u16* __restrict__ V,
    void* __restrict__ Out, float* __restrict__ LSE, int Nq, int Nk, int n_qtiles, float c) {
    using T = Tile<D>;
    constexpr uint32_t ROW_BYTES = D * 2;
    __shared__ __attribute__((aligned(16))) u16 Ks[T::K_ELEMS];
    __shared__ __attribute__((aligned(16))) u16 Vt[T::V_ELEMS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int col = lane & 31;     // query within the wave's 32
    const int half = lane >> 5;    // which 8-element k group of the MFMA operands

    int bh, qt;
    tile_of_block(blockIdx.x, gridDim.x, n_qtiles, CAUSAL, bh, qt);
    const int q0 = qt * BM;
    const int off = Nk - Nq;       // causal: key j visible to query i iff j <= i + off

    const u16* Qh = Q + (size_t)bh * Nq * D;
    const u16* Kh = K + (size_t)bh * Nk * D;
    const u16* Vh = V + (size_t)bh * Nk * D;

    // A negative scale is folded into Q's sign (exact for bf16) so that the
    // softmax below always sees c >= 0.
    const uint32_t qflip = (c < 0.0f) ? 0x80008000u : 0u;
    c = fabsf(c);

    // ---- a1: Q fragment for this lane's query, all of d, kept in registers.
    // Rows past Nq read as zeros (buffer bounds) and are never stored.
    const int qrow = q0 + wave * 32 + col;
    bf16x8 qf[D / 16];
    {
        const auto rq = make_rsrc(Qh, (uint32_t)Nq * ROW_BYTES);
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
            uint4 w = buffer_load16(rq, (uint32_t)qrow * ROW_BYTES + s * 32 + half * 16);
            w.x ^= qflip; w.y ^= qflip; w.z ^= qflip; w.w ^= qflip;
            qf[s] = __builtin_bit_cast(bf16x8, w);
        }
    }

    // Key range this tile of queries needs.
    int kv_end = Nk;
    if (CAUSAL) kv_end = min(Nk, q0 + BM + off);
    const int n_kt = (kv_end + BN - 1) / BN;
    const int wave_q_first = q0 + wave * 32;
    const int wave_q_last = wave_q_first + 31;

    // ---- a2: register staging of one K/V tile (global -> regs -> LDS).
    // Per-thread byte offsets inside a tile are fixed; each tile only moves the
    // buffer base, and keys past Nk read as zeros.
    uint4 kreg[T::K_PASSES];
    uint4 vreg0, vreg1, vreg2, vreg3;
    const bool v_loader = tid < T::V_THREADS;
    const int v_kg = tid % (BN / 4);      // keys 4*v_kg .. 4*v_kg+3
    const int v_dg = tid / (BN / 4);      // dv 8*v_dg .. 8*v_dg+7
    const uint32_t v_off = (uint32_t)(4 * v_kg) * ROW_BYTES + v_dg * 16;

    auto load_tile = [&](int kt) {
        const int kbase = kt * BN;
        const uint32_t bytes = (uint32_t)(Nk - kbase) * ROW_BYTES;
        const auto rk = make_rsrc(Kh + (size_t)kbase * D, bytes);
#pragma unroll
        for (int p = 0; p < T::K_PASSES; ++p)
            kreg[p] = buffer_load16(rk, (uint32_t)(tid + p * THREADS) * 16);
        if (v_loader) {
            const auto rv = make_rsrc(Vh + (size_t)kbase * D, bytes);
            vreg0 = buffer_load16(rv, v_off);
            vreg1 = buffer_load16(rv, v_off + ROW_BYTES);
            vreg2 = buffer_load16(rv, v_off + 2 * ROW_BYTES);
            vreg3 = buffer_load16(rv, v_off + 3 * ROW_BYTES);
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < T::K_PASSES; ++p) {
            const int idx = tid + p * THREADS;
            const int row = idx / (D / 8), ch = idx % (D / 8);
            *reinterpret_cast<uint4*>(&Ks[row * T::KSTRIDE + ch * 8]) = kreg[p];
        }
        if (v_loader) {
            // transpose 4 keys x 8 dv into V^T rows: element (dv, key)
            u16* dst = &Vt[(v_dg * 8) * T::VSTRIDE + 4 * v_kg];
            auto put = [&](int j, uint32_t a, uint32_t b, uint32_t cc, uint32_t d, bool hi) {
                uint2 w;
                if (!hi) {
                    w.x = __builtin_amdgcn_perm(b, a, 0x05040100u);
                    w.y = __builtin_amdgcn_perm(d, cc, 0x05040100u);
                } else {
                    w.x = __builtin_amdgcn_perm(b, a, 0x07060302u);
                    w.y = __builtin_amdgcn_perm(d, cc, 0x07060302u);
                }
                *reinterpret_cast<uint2*>(dst + j * T::VSTRIDE) = w;
            };
            put(0, vreg0.x, vreg1.x, vreg2.x, vreg3.x, false);
            put(1, vreg0.x, vreg1.x, vreg2.x, vreg3.x, true);
            put(2, vreg0.y, vreg1.y, vreg2.y, vreg3.y, false);
            put(3, vreg0.y, vreg1.y, vreg2.y, vreg3.y, true);
            put(4, vreg0.z, vreg1.z, vreg2.z, vreg3.z, false);
            put(5, vreg0.z, vreg1.z, vreg2.z, vreg3.z, true);
            put(6, vreg0.w, vreg1.w, vreg2.w, vreg3.w, false);
            put(7, vreg0.w, vreg1.w, vreg2.w, vreg3.w, true);
        }
    };

    f32x16 oacc[D / 32];
#pragma unroll
    for (int b = 0; b < D / 32; ++b) oacc[b] = f32x16{};
    float m_run = kNegInf;   // running max, log2 units (scores * c)
    float l_run = 0.0f;      // partial denominator over this half-wave's keys

    // One key tile for this wave: a3..a6.  MASK selects the variant for tiles
    // that contain keys past Nk or past some query's diagonal.
    auto compute_tile = [&](const int kbase, auto mask_tag) {
        constexpr bool MASK = decltype(mask_tag)::value;

        // ---- a3: S^T tile (64 keys x 32 queries) = K_tile . Q^T on MFMA.
        f32x16 sacc[BN / 32];
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb) sacc[kb] = f32x16{};
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
#pragma unroll
            for (int kb = 0; kb < BN / 32; ++kb) {
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(
                    &Ks[(kb * 32 + col) * T::KSTRIDE + s * 16 + half * 8]);
                sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], sacc[kb], 0, 0, 0);
            }
        }
        if constexpr (MASK) {
#pragma unroll
            for (int kb = 0; kb < BN / 32; ++kb) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = kbase + kb * 32 + (i >> 2) * 8 + half * 4 + (i & 3);
                    const bool masked = key >= Nk || (CAUSAL && key > qrow + off);
                    if (masked) sacc[kb][i] = kNegInf;
                }
            }
        }

        // ---- a4: tile row max (in-lane, then across the two half-waves).
        float mx = kNegInf;
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kb][i]);
        mx = half_max(mx);
        const float mt = (MASK && mx == kNegInf) ? kNegInf : mx * c;

        // Raise the reference maximum only when the tile exceeds it by the slack.
        if (wave_any(mt > m_run + kRescaleSlack)) {
            const float m_new = fmaxf(m_run, mt);
            const float alpha = (m_run == kNegInf) ? 0.0f : exp2_hw(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int b = 0; b < D / 32; ++b) oacc[b] *= alpha;
            m_run = m_new;
        }

        // ---- a5: weights p = 2^(s c - m), partial row sum, pack to bf16.
        const float neg_m = -m_run;
        bf16x8 pb[BN / 16];
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float p = exp2_hw(__builtin_fmaf(sacc[kb][i], c, neg_m));
                if constexpr (MASK) p = (sacc[kb][i] == kNegInf) ? 0.0f : p;
                l_run += p;
                pb[kb * 2 + (i >> 3)][i & 7] = (__bf16)p;
            }
        }

        // ---- a6: O^T += V^T . P^T on MFMA.  Chunk cc covers keys
        // 16cc + 4*half + {0..3} and 16cc + 8 + 4*half + {0..3}, matching pb.
#pragma unroll
        for (int cc = 0; cc < BN / 16; ++cc) {
#pragma unroll
            for (int b = 0; b < D / 32; ++b) {
                const u16* vrow = &Vt[(b * 32 + col) * T::VSTRIDE + cc * 16 + half * 4];
                const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
                const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 8);
                const uint4 w = make_uint4(lo.x, lo.y, hi.x, hi.y);
                oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, w), pb[cc], oacc[b], 0, 0, 0);
            }
        }
    };

    load_tile(0);
    for (int kt = 0; kt < n_kt; ++kt) {
        __syncthreads();            // previous tile fully consumed
        store_tile();
        __syncthreads();            // tile visible to all waves
        if (kt + 1 < n_kt) load_tile(kt + 1);

        const int kbase = kt * BN;
        if (CAUSAL && kbase > wave_q_last + off) continue;   // tile fully masked for this wave
        const bool need_mask = (kbase + BN > Nk) || (CAUSAL && kbase + BN - 1 > wave_q_first + off);
        if (need_mask)
            compute_tile(kbase, std::true_type{});
        else
            compute_tile(kbase, std::false_type{});
    }

    // ---- a7: epilogue, O = acc / l: the only device-memory write.
    const float l_tot = half_sum(l_run);
    const float inv = 1.0f / l_tot;
    if (qrow < Nq) {
        const size_t obase = ((size_t)bh * Nq + qrow) * D;
#pragma unroll
        for (int b = 0; b < D / 32; ++b) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int dv = b * 32 + g * 8 + half * 4;
                const float o0 = oacc[b][g * 4 + 0] * inv, o1 = oacc[b][g * 4 + 1] * inv;
                const float o2 = oacc[b][g * 4 + 2] * inv, o3 = oacc[b][g * 4 + 3] * inv;
                if (OUT_BF16) {
                    uint2 w = make_uint2(pack_bf16x2(o0, o1), pack_bf16x2(o2, o3));
                    *reinterpret_cast<uint2*>(static_cast<u16*>(Out) + obase + dv) = w;
                } else {
                    *reinterpret_cast<float4*>(static_cast<float*>(Out) + obase + dv) =
                        make_float4(o0, o1, o2, o3);
                }
            }
        }
        if (LSE != nullptr && half == 0)
            LSE[(size_t)bh * Nq + qrow] = (m_run + __log2f(l_tot)) * kLn2;
    }
}

template <int D, bool CAUSAL, bool OUT_BF16>
hipError_t launch(const Problem& p, hipStream_t stream) {
    const int n_qtiles = (p.nq + BM - 1) / BM;
    const long long blocks = (long long)p.bh * n_qtiles;
    const float c = p.scale * kLog2e;
    return launch_kernel(prefill_bf16_kernel<D, CAUSAL, OUT_BF16>, dim3((unsigned)blocks),
                         dim3(THREADS), stream, static_cast<const u16*>(p.q),
                         static_cast<const u16*>(p.k), static_cast<const u16*>(p.v), p.o, p.lse,
                         p.nq, p.nk, n_qtiles, c);
}

template <int D>
hipError_t launch_d(const Problem& p, hipStream_t stream) {
    if (p.causal)
        return p.out_bf16 ? launch<D, true, true>(p, stream) : launch<D, true, false>(p, stream);
    return p.out_bf16 ? launch<D, false, true>(p, stream) : launch<D, false, false>(p, stream);
}

}  // namespace

static_assert(BM == kPrefillBf16RowsPerBlock, "row tile mismatch");

hipError_t launch_prefill_bf16(const Problem& p, hipStream_t stream) {
    if (p.d == 64) return launch_d<64>(p, stream);
    if (p.d == 128) return launch_d<128>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
