// Backward pass of fused attention for bf16 inputs on gfx950 matrix cores:
// dQ, dK and dV for a given dO, recomputing the weights from the forward's
// LSE (no score or weight matrix is ever stored, as in the forward).
//
// With s = <q_i, k_j>, c = scale * log2(e) and lse2_i = LSE_i * log2(e):
//   P_ij  = 2^(s_ij c - lse2_i)              (the forward's softmax weights)
//   dP_ij = <dO_i, v_j>
//   D_i   = <dO_i, O_i> = sum_j P_ij dP_ij
//   dS_ij = P_ij (dP_ij - D_i)               (softmax Jacobian)
//   dQ_i  = scale * sum_j dS_ij k_j,   dK_j = scale * sum_i dS_ij q_i,
//   dV_j  = sum_i P_ij dO_i
// which is the chain rule through the softmax the paper leaves to its Stage 5.
//
// Three kernels:
//  * bwd_rowdot: D_i from dO and O (fp32).
//  * bwd_dq: one item = 256 queries of one (b, h); K and V stream through LDS
//    in 64-key stages.  S^T = K Q^T and dP^T = V dO^T on the MFMA (K and V
//    rows as A operands, Q and dO fragments held in registers as in the
//    forward), dS^T in registers, dQ^T += K^T dS^T with K^T from transposing
//    LDS reads of the same K stage.
//  * bwd_dkdv_pair: one item = 128 keys of one (b, h); Q, dO, LSE and D
//    stream through LDS in 64-query stages.  S = Q K^T and dP = dO V^T (Q and
//    dO rows as A operands, K or V fragments in registers), so a lane holds
//    one key; dV^T += dO^T P and dK^T += Q^T dS with dO^T and Q^T from
//    transposing reads.  The two halves of that work go to two waves of the
//    same SIMD (the weights P pass between them through LDS), so the vector
//    work of one overlaps the matrix products of the other.  Every lane owns
//    its key's rows of dK or dV: no atomics, and the results are
//    deterministic.
// P and dS are rounded to bf16 for the matrix products (fp32 accumulation);
// dS is formed from the bf16-rounded P.
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "prefill_bf16_common.h"

namespace moa {
namespace {

using namespace pf;

constexpr int SUB = 32;   // queries (bwd_dkdv) or keys (bwd_dq) per step

// ---- D_i = <dO_i, O_i>: 16 lanes per row (8 elements each), 4 rows per wave.
template <int D, bool O_BF16>
__global__ __launch_bounds__(256) void bwd_rowdot_kernel(const u16* __restrict__ dO,
                                                         const void* __restrict__ O,
                                                         float* __restrict__ Dsum, long long rows) {
    constexpr int LPR = D / 8;
    const long long row = (long long)blockIdx.x * (256 / LPR) + threadIdx.x / LPR;
    const int e0 = (threadIdx.x % LPR) * 8;
    float acc = 0.0f;
    if (row < rows) {
        const uint4 g = *reinterpret_cast<const uint4*>(dO + row * D + e0);
        const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
        float o[8];
        if (O_BF16) {
            const uint4 h = *reinterpret_cast<const uint4*>(static_cast<const u16*>(O) + row * D + e0);
            const uint32_t hw[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                o[2 * j] = __uint_as_float(hw[j] << 16);
                o[2 * j + 1] = __uint_as_float(hw[j] & 0xffff0000u);
            }
        } else {
            const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(O) + row * D + e0);
            const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(O) + row * D + e0 + 4);
            o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w; o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            acc = __builtin_fmaf(__uint_as_float(gw[j] << 16), o[2 * j], acc);
            acc = __builtin_fmaf(__uint_as_float(gw[j] & 0xffff0000u), o[2 * j + 1], acc);
        }
    }
#pragma unroll
    for (int m = 1; m < LPR; m <<= 1) acc += __shfl_xor(acc, m);
    if (row < rows && (threadIdx.x % LPR) == 0) Dsum[row] = acc;
}

// Per-lane LDS addresses shared by both kernels (the stage layout of the
// forward: 64 rows of D bf16, 16-byte chunks XOR-swizzled per row).
template <int D>
struct TileAddr {
    uint32_t row[D / 16];      // A operand of a row-major stage: row col (+32 u), chunk 2s + half
    uint32_t tr[D / 32][2];    // transposing reads: D-block b, lo / hi row quads
    __device__ __forceinline__ TileAddr(int lane) {
        constexpr uint32_t RB = Cfg<D>::ROW_BYTES;
        const int col = lane & 31, half = lane >> 5;
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
            row[s] = (uint32_t)col * RB + (uint32_t)(((2 * s + half) ^ swz<D>(col)) * 16);
        const int g = lane >> 4, j = (lane >> 2) & 3, q = lane & 3;
#pragma unroll
        for (int b = 0; b < D / 32; ++b)
#pragma unroll
            for (int h8 = 0; h8 < 2; ++h8) {
                const int r = 4 * (g >> 1) + j + 8 * h8;
                const int dv = dv_of<D>(b, 16 * (g & 1) + 4 * q);
                tr[b][h8] = (uint32_t)r * RB + (uint32_t)((((dv >> 3) ^ swz<D>(r)) * 16) + (dv & 7) * 2);
            }
    }
};

// MFMA A operand from a stage: rows 32u + (lane % 32), contraction chunk s.
template <int D>
__device__ __forceinline__ bf16x8 stage_rows(const unsigned char* st, const TileAddr<D>& a, int u, int s) {
    return *reinterpret_cast<const bf16x8*>(st + a.row[s] + u * 32 * Cfg<D>::ROW_BYTES);
}
// MFMA A operand of the transposed stage: D-block b, 16-row chunk cc.
template <int D>
__device__ __forceinline__ bf16x8 stage_tr(const unsigned char* st, const TileAddr<D>& a, int b, int cc) {
    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(st + a.tr[b][0] + cc * 16 * Cfg<D>::ROW_BYTES));
    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(st + a.tr[b][1] + cc * 16 * Cfg<D>::ROW_BYTES));
    const v4s both[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, both);
}

// Packs an fp32 accumulator (16 values) into two bf16x8 MFMA B operands in the
// key (or query) order of the transposing reads: chunk c2 takes elements
// 8 c2 .. 8 c2 + 7.
__device__ __forceinline__ void pack16(const float (&x)[16], bf16x8 (&pb)[2]) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        u32x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const bf16x2 pp = {(__bf16)x[8 * g + 2 * j], (__bf16)x[8 * g + 2 * j + 1]};
            w[j] = __builtin_bit_cast(uint32_t, pp);
        }
        pb[g] = __builtin_bit_cast(bf16x8, w);
    }
}

// A direct-to-LDS 16-byte load (buffer_load_dwordx4 ... lds) as inline
// assembly, invisible to the compiler's wait-count tracking (whose aliasing
// model cannot tell the slots of one LDS ring apart and would wait for every
// load before any read of the ring).  The
// caller waits for it itself (s_waitcnt vmcnt, then a barrier) before any wave
// reads the data; loads complete in issue order, so the compiler's own waits
// for later loads stay correct.  `rsrc` holds the four descriptor words (see
// rsrc_words), `lds_addr` the wave-uniform LDS byte address.
__device__ __forceinline__ u32x4 rsrc_words(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return u32x4{(uint32_t)a, (uint32_t)(a >> 32) & 0xffffu, bytes, 0x00020000u};
}
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p);
}
// M0 is listed as clobbered: clang warns that it does not preserve reserved
// registers around the statement; the kernels of this file set M0 nowhere
// else (their assembly has no other M0 write).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void buffer_load16_to_lds_untracked(u32x4 rsrc, uint32_t lds_addr, uint32_t voffset) {
    const u32x4 r = {(uint32_t)__builtin_amdgcn_readfirstlane(rsrc[0]), (uint32_t)__builtin_amdgcn_readfirstlane(rsrc[1]),
                     (uint32_t)__builtin_amdgcn_readfirstlane(rsrc[2]), (uint32_t)__builtin_amdgcn_readfirstlane(rsrc[3])};
    const uint32_t m = (uint32_t)__builtin_amdgcn_readfirstlane(lds_addr);
    // One wait state between the M0 write and the load that reads it.
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(m), "v"(voffset), "s"(r) : "memory", "m0");
}
#pragma clang diagnostic pop

// Direct-to-LDS stage loads (untracked: the caller waits with vmcnt and a
// barrier): lane l of the i-th load of wave w fills slot S = (w*LPS + i)*64
// + l of the stage, which holds logical chunk (S % CHUNKS) ^ swz(row) of row
// S / CHUNKS (the forward's swizzled layout).
template <int D, int NW>
struct DmaStager {
    static constexpr int LPS = Cfg<D>::TILE_BYTES / (NW * 1024);
    static_assert(Cfg<D>::TILE_BYTES % (NW * 1024) == 0, "a stage must split into wave loads");
    uint32_t goff[LPS];
    uint32_t lds_off;        // this wave's first 1 KB of a stage
    __device__ __forceinline__ DmaStager(int wave, int lane) {
        lds_off = (uint32_t)wave * LPS * 1024u;
#pragma unroll
        for (int i = 0; i < LPS; ++i) {
            const int slot = (wave * LPS + i) * 64 + lane;
            const int row = slot / Cfg<D>::CHUNKS, p = slot % Cfg<D>::CHUNKS;
            goff[i] = (uint32_t)row * Cfg<D>::ROW_BYTES + (uint32_t)((p ^ swz<D>(row)) * 16);
        }
    }
    // Rows j*64 .. j*64 + 63 of a head slice of `n` rows into `stage`; rows
    // past n are zero.
    __device__ __forceinline__ void issue(const u16* head, int n, int j, unsigned char* stage) const {
        const int r0 = min(j * BN, n);
        const u32x4 r = rsrc_words(head + (size_t)r0 * D, (uint32_t)(n - r0) * Cfg<D>::ROW_BYTES);
        const uint32_t base = lds_address(stage) + lds_off;
#pragma unroll
        for (int i = 0; i < LPS; ++i) buffer_load16_to_lds_untracked(r, base + i * 1024u, goff[i]);
    }
};

template <int D, bool OUT_BF16>
__device__ __forceinline__ void store_rows16(void* out, size_t row_base, int half, const f32x16 (&acc)[D / 32],
                                             float mul) {
#pragma unroll
    for (int b = 0; b < D / 32; ++b)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int dv = dv_of<D>(b, g * 8 + half * 4);
            const float o0 = acc[b][g * 4 + 0] * mul, o1 = acc[b][g * 4 + 1] * mul;
            const float o2 = acc[b][g * 4 + 2] * mul, o3 = acc[b][g * 4 + 3] * mul;
            if (OUT_BF16) {
                *reinterpret_cast<uint2*>(static_cast<u16*>(out) + row_base + dv) =
                    make_uint2(pack_bf16x2(o0, o1), pack_bf16x2(o2, o3));
            } else {
                *reinterpret_cast<float4*>(static_cast<float*>(out) + row_base + dv) =
                    make_float4(o0, o1, o2, o3);
            }
        }
}

// ---- dQ: 8 waves x 32 queries; K and V stages of 64 keys.
constexpr int DQ_WAVES = 8;
constexpr int DQ_THREADS = DQ_WAVES * 64;
constexpr int DQ_BM = DQ_WAVES * 32;

template <int D, bool CAUSAL, bool OUT_BF16>
__global__ __launch_bounds__(DQ_THREADS, 1) void bwd_dq_kernel(
    const u16* __restrict__ Q, const u16* __restrict__ K, const u16* __restrict__ V,
    const u16* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ Dsum,
    void* __restrict__ dQ, int Nq, int Nk, int n_bh, int n_qtiles, float c, float scale) {
    using C = Cfg<D>;
    constexpr uint32_t RB = C::ROW_BYTES;
    __shared__ __attribute__((aligned(1024))) unsigned char k_r0[C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char k_r1[C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char v_r0[C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char v_r1[C::TILE_BYTES];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int col = lane & 31, half = lane >> 5;
    const int off = Nk - Nq;
    const TileAddr<D> ta(lane);
    const DmaStager<D, DQ_WAVES> stg(wave, lane);

    for (int item = 0;; ++item) {
        int bh, qt;
        if (!item_of(blockIdx.x, item, gridDim.x, n_bh, n_qtiles, CAUSAL, bh, qt)) break;
        const int q0 = qt * DQ_BM;
        const int qrow = q0 + wave * 32 + col;
        const u16* Kh = K + (size_t)bh * Nk * D;
        const u16* Vh = V + (size_t)bh * Nk * D;

        // Q and dO fragments of this lane's query (B operands), its LSE and D.
        bf16x8 qf[D / 16], gf[D / 16];
        {
            const auto rq = make_rsrc(Q + (size_t)bh * Nq * D, (uint32_t)Nq * RB);
            const auto rg = make_rsrc(dO + (size_t)bh * Nq * D, (uint32_t)Nq * RB);
#pragma unroll
            for (int s = 0; s < D / 16; ++s) {
                qf[s] = __builtin_bit_cast(bf16x8, buffer_load16(rq, (uint32_t)qrow * RB + s * 32 + half * 16));
                gf[s] = __builtin_bit_cast(bf16x8, buffer_load16(rg, (uint32_t)qrow * RB + s * 32 + half * 16));
            }
        }
        const bool row_ok = qrow < Nq;
        const float lse2 = row_ok ? LSE[(size_t)bh * Nq + qrow] * kLog2e : 0.0f;
        const float dsum = row_ok ? Dsum[(size_t)bh * Nq + qrow] : 0.0f;

        const int kv_end = CAUSAL ? min(Nk, q0 + DQ_BM + off) : Nk;
        const int n_sub = (kv_end + SUB - 1) / SUB;
        const int n_stages = (n_sub + 1) / 2;
        const int wave_q_first = q0 + wave * 32;
        int n_w = n_sub;
        if (wave_q_first >= Nq) n_w = 0;
        else if (CAUSAL) n_w = min(n_sub, (wave_q_first + 31 + off) / SUB + 1);

        f32x16 acc[D / 32];
#pragma unroll
        for (int b = 0; b < D / 32; ++b) acc[b] = f32x16{};

        // One step of 32 keys (half u of the stage in ks / vs, global step t).
        auto step = [&](const unsigned char* ks, const unsigned char* vs, int u, int t)
                        __attribute__((always_inline)) {
            f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
            for (int k = 0; k < D / 16; ++k) {
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_rows<D>(ks, ta, u, k), qf[k], s, 0, 0, 0);
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_rows<D>(vs, ta, u, k), gf[k], dp, 0, 0, 0);
            }
            const int kbase = t * SUB;
            const bool need_mask = (kbase + SUB > Nk) || (CAUSAL && kbase + SUB - 1 > wave_q_first + off);
            float ds[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float t = __builtin_fmaf(s[i], c, -lse2);
                if (need_mask) {
                    const int key = kbase + (i >> 2) * 8 + half * 4 + (i & 3);
                    if (key >= Nk || (CAUSAL && key > qrow + off)) t = kNegInf;
                }
                ds[i] = exp2_hw(t) * (dp[i] - dsum);
            }
            bf16x8 dsb[2];
            pack16(ds, dsb);
#pragma unroll
            for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
                for (int b = 0; b < D / 32; ++b)
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_tr<D>(ks, ta, b, 2 * u + c2), dsb[c2],
                                                                     acc[b], 0, 0, 0);
        };

        // Stage iteration j: K(j), V(j) in slot j & 1.  Right after the
        // barrier the loads of K(j+1), V(j+1) start into the other slot,
        // whose readers (iteration j - 1) are done; each wave waits for its
        // own loads before the next barrier.
        stg.issue(Kh, Nk, 0, k_r0);
        stg.issue(Vh, Nk, 0, v_r0);
        for (int j = 0; j < n_stages; ++j) {
            unsigned char* ks = (j & 1) ? k_r1 : k_r0;
            unsigned char* vs = (j & 1) ? v_r1 : v_r0;
            wait_vmcnt<0>();
            wait_lgkmcnt0();
            barrier_no_fence();
            if (j + 1 < n_stages) {
                stg.issue(Kh, Nk, j + 1, (j & 1) ? k_r0 : k_r1);
                stg.issue(Vh, Nk, j + 1, (j & 1) ? v_r0 : v_r1);
            }
            if (2 * j < n_w) step(ks, vs, 0, 2 * j);
            if (2 * j + 1 < n_w) step(ks, vs, 1, 2 * j + 1);
        }
        wait_lgkmcnt0();
        barrier_no_fence();
        if (row_ok) store_rows16<D, OUT_BF16>(dQ, ((size_t)bh * Nq + qrow) * D, half, acc, scale);
    }
}

// ---- dK, dV with two waves per SIMD: 8 waves, 128 keys per item.  Wave w
// < 4 (role A) owns keys 32w .. 32w + 31 of the item for dV: S = Q K^T, the
// weights P (exponentials), dV^T += dO^T P, and P handed to its partner
// through LDS as bf16.  Wave w + 4 (role B, on the same SIMD) owns the same
// keys for dK: dP = dO V^T, dS = P (dP - D) with the partner's P, dK^T +=
// Q^T dS.  The matrix work of a step splits evenly between the two waves and
// nothing is computed twice; B runs one 64-query stage behind A, so the LDS
// ring holds three Q / dO stages and two stages of exchanged weights.
constexpr int KV2_WAVES = 8;
constexpr int KV2_THREADS = KV2_WAVES * 64;
constexpr int KV2_BN = 4 * 32;   // keys per item
constexpr int KV2_RING = 3;      // Q / dO stages in LDS

template <int D, bool CAUSAL, bool OUT_BF16>
__global__ __launch_bounds__(KV2_THREADS, 1) void bwd_dkdv_pair_kernel(
    const u16* __restrict__ Q, const u16* __restrict__ K, const u16* __restrict__ V,
    const u16* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ Dsum,
    void* __restrict__ dK, void* __restrict__ dV, int Nq, int Nk, int n_bh, int n_ktiles, float c,
    float scale) {
    using C = Cfg<D>;
    constexpr uint32_t RB = C::ROW_BYTES;
    __shared__ __attribute__((aligned(1024))) unsigned char q_r[KV2_RING][C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char g_r[KV2_RING][C::TILE_BYTES];
    // Exchanged weights: [stage parity][key block][32-query half][chunk c2][lane] x 16 bytes.
    __shared__ __attribute__((aligned(1024))) uint4 p_x[2][4][2][2][64];
    __shared__ __attribute__((aligned(16))) float l_r[KV2_RING][2][BN];   // [slot][lse2, D][query]

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int role = wave >> 2, kb = wave & 3;   // role 0: P and dV; role 1: dS and dK
    const int col = lane & 31, half = lane >> 5;
    const int off = Nk - Nq;
    const TileAddr<D> ta(lane);
    const DmaStager<D, KV2_WAVES> stg(wave, lane);

    for (int item = 0;; ++item) {
        int bh, rt;
        if (!item_of(blockIdx.x, item, gridDim.x, n_bh, n_ktiles, CAUSAL, bh, rt)) break;
        // Causal key tiles cost most at the start of the sequence: the
        // heaviest-first rank order of item_of is reversed here.
        const int kt = CAUSAL ? n_ktiles - 1 - rt : rt;
        const int k0 = kt * KV2_BN;
        const int krow = k0 + kb * 32 + col;
        const bool key_ok = krow < Nk;
        const u16* Qh = Q + (size_t)bh * Nq * D;
        const u16* Gh = dO + (size_t)bh * Nq * D;
        const float* Lh = LSE + (size_t)bh * Nq;
        const float* Dh = Dsum + (size_t)bh * Nq;

        // K (role A) or V (role B) fragment of this lane's key: B operands.
        bf16x8 kvf[D / 16];
        {
            const auto r = make_rsrc((role == 0 ? K : V) + (size_t)bh * Nk * D, (uint32_t)Nk * RB);
#pragma unroll
            for (int s = 0; s < D / 16; ++s)
                kvf[s] = __builtin_bit_cast(bf16x8, buffer_load16(r, (uint32_t)krow * RB + s * 32 + half * 16));
        }

        // Queries that see any key of the tile (query i sees key j iff
        // j <= i + off), in 64-query stages; the block's first needed step.
        const int q_lo = CAUSAL ? max(0, k0 - off) : 0;
        const int st0 = q_lo / BN;
        const int n_stages = (Nq + BN - 1) / BN - st0;
        const int blk_k_first = k0 + kb * 32;
        const int t_first = CAUSAL ? max(0, blk_k_first - off) / SUB : 0;   // global 32-query step
        const bool blk_live = blk_k_first < Nk;

        f32x16 acc[D / 32];          // dV^T (role A) or dK^T (role B)
#pragma unroll
        for (int b = 0; b < D / 32; ++b) acc[b] = f32x16{};

        // Role A, step u of stage js: weights of 32 queries x this lane's key.
        auto step_a = [&](const unsigned char* qs, const unsigned char* gs, const float* ls, uint4* px,
                          int u, int t) __attribute__((always_inline)) {
            f32x16 s = f32x16{};
#pragma unroll
            for (int k = 0; k < D / 16; ++k)
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_rows<D>(qs, ta, u, k), kvf[k], s, 0, 0, 0);
            const int qbase = t * SUB;
            const bool need_mask = (qbase + SUB > Nq) || (CAUSAL && qbase < blk_k_first + 31 - off);
            float p[16];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int m0 = 32 * u + 8 * g + 4 * half;   // stage-local query of element 4g
                const float4 l4 = *reinterpret_cast<const float4*>(ls + m0);
                const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = 4 * g + r;
                    float x = __builtin_fmaf(s[i], c, -lv[r]);
                    if (need_mask) {
                        const int qi = qbase + 8 * g + 4 * half + r;
                        if (qi >= Nq || (CAUSAL && krow > qi + off)) x = kNegInf;
                    }
                    p[i] = exp2_hw(x);
                }
            }
            bf16x8 pb[2];
            pack16(p, pb);
#pragma unroll
            for (int c2 = 0; c2 < 2; ++c2) px[c2 * 64 + lane] = __builtin_bit_cast(uint4, pb[c2]);
#pragma unroll
            for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
                for (int b = 0; b < D / 32; ++b)
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_tr<D>(gs, ta, b, 2 * u + c2), pb[c2],
                                                                     acc[b], 0, 0, 0);
        };

        // Role B, step u of stage js: dS from the partner's weights.
        auto step_b = [&](const unsigned char* qs, const unsigned char* gs, const float* dsv, const uint4* px,
                          int u) __attribute__((always_inline)) {
            f32x16 dp = f32x16{};
#pragma unroll
            for (int k = 0; k < D / 16; ++k)
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_rows<D>(gs, ta, u, k), kvf[k], dp, 0, 0, 0);
            const uint4 w0 = px[lane], w1 = px[64 + lane];
            const uint32_t pw[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
            float ds[16];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int m0 = 32 * u + 8 * g + 4 * half;
                const float4 d4 = *reinterpret_cast<const float4*>(dsv + m0);
                const float dvv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = 4 * g + r;
                    const float pi = (i & 1) ? bf16hi_to_f32(pw[i >> 1]) : bf16lo_to_f32(pw[i >> 1]);
                    ds[i] = pi * (dp[i] - dvv[r]);
                }
            }
            bf16x8 dsb[2];
            pack16(ds, dsb);
#pragma unroll
            for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
                for (int b = 0; b < D / 32; ++b)
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(stage_tr<D>(qs, ta, b, 2 * u + c2), dsb[c2],
                                                                     acc[b], 0, 0, 0);
        };

        // LSE and D of a stage's 64 queries: one float per lane of waves 0
        // and 1 (zero past Nq), stored one iteration after the load.
        auto load_ld = [&](int js, float& x) __attribute__((always_inline)) {
            const int qi = js * BN + lane;
            x = 0.0f;
            if (wave < 2 && qi < Nq) x = (wave == 0) ? Lh[qi] : Dh[qi];
        };

        // Iteration j: stage st0 + j is in the ring; role A works on it,
        // role B on the stage before (whose weights A wrote in iteration
        // j - 1).  Right after the barrier the loads of stage j + 1 start
        // into the slot whose last reader (role B, iteration j - 1) is done,
        // and each wave waits for its own loads before the next barrier.
        float sx;
        stg.issue(Qh, Nq, st0, q_r[0]);
        stg.issue(Gh, Nq, st0, g_r[0]);
        load_ld(st0, sx);
        for (int j = 0; j <= n_stages; ++j) {
            const int js = st0 + j;
            const int slot = j % KV2_RING;
            if (j < n_stages && wave < 2) l_r[slot][wave][lane] = (wave == 0) ? sx * kLog2e : sx;
            wait_vmcnt<0>();
            wait_lgkmcnt0();
            barrier_no_fence();
            if (j + 1 < n_stages) {
                const int ns = (j + 1) % KV2_RING;
                stg.issue(Qh, Nq, js + 1, q_r[ns]);
                stg.issue(Gh, Nq, js + 1, g_r[ns]);
                load_ld(js + 1, sx);
            }
            if (!blk_live) continue;
            if (role == 0) {
                if (j < n_stages) {
#pragma unroll
                    for (int u = 0; u < 2; ++u)
                        if (2 * js + u >= t_first)
                            step_a(q_r[slot], g_r[slot], l_r[slot][0], &p_x[j & 1][kb][u][0][0], u, 2 * js + u);
                }
            } else if (j >= 1) {
                const int ps = (j - 1) % KV2_RING;
#pragma unroll
                for (int u = 0; u < 2; ++u)
                    if (2 * (js - 1) + u >= t_first)
                        step_b(q_r[ps], g_r[ps], l_r[ps][1], &p_x[(j - 1) & 1][kb][u][0][0], u);
            }
        }
        wait_lgkmcnt0();
        barrier_no_fence();
        if (key_ok) {
            const size_t base = ((size_t)bh * Nk + krow) * D;
            if (role == 0) store_rows16<D, OUT_BF16>(dV, base, half, acc, 1.0f);
            else store_rows16<D, OUT_BF16>(dK, base, half, acc, scale);
        }
    }
}

template <typename Kern>
int resident_per_cu(Kern kernel, int threads) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess) n = 1;
    return n > 0 ? n : 1;
}

template <int D, bool CAUSAL, bool OUT_BF16>
hipError_t launch(const BwdProblem& p, hipStream_t stream) {
    int cus = 0;
    hipError_t e = device_cus(stream, cus);
    if (e != hipSuccess) return e;
    const long long rows = (long long)p.bh * p.nq;
    // D_i, then dQ (both have nothing to do without queries)
    if (rows > 0) {
        const unsigned grid = (unsigned)((rows + (256 / (D / 8)) - 1) / (256 / (D / 8)));
        e = p.o_bf16 ? launch_kernel(bwd_rowdot_kernel<D, true>, dim3(grid), dim3(256), stream,
                                     static_cast<const u16*>(p.dout), p.o, p.dsum, rows)
                     : launch_kernel(bwd_rowdot_kernel<D, false>, dim3(grid), dim3(256), stream,
                                     static_cast<const u16*>(p.dout), p.o, p.dsum, rows);
        if (e != hipSuccess) return e;
    }
    const float c = p.scale * kLog2e;
    if (rows > 0) {
        auto kernel = bwd_dq_kernel<D, CAUSAL, OUT_BF16>;
        static const int per_cu = resident_per_cu(kernel, DQ_THREADS);
        const int n_qt = (p.nq + DQ_BM - 1) / DQ_BM;
        const long long items = (long long)p.bh * n_qt;
        const unsigned grid = (unsigned)std::min<long long>(items, (long long)cus * per_cu);
        e = launch_kernel(kernel, dim3(grid), dim3(DQ_THREADS), stream, static_cast<const u16*>(p.q),
                          static_cast<const u16*>(p.k), static_cast<const u16*>(p.v),
                          static_cast<const u16*>(p.dout), p.lse, static_cast<const float*>(p.dsum),
                          p.dq, p.nq, p.nk, p.bh, n_qt, c, p.scale);
        if (e != hipSuccess) return e;
    }
    // dK, dV (zero when there are no queries)
    {
        auto kernel = bwd_dkdv_pair_kernel<D, CAUSAL, OUT_BF16>;
        static const int per_cu = resident_per_cu(kernel, KV2_THREADS);
        const int n_kt = (p.nk + KV2_BN - 1) / KV2_BN;
        const long long items = (long long)p.bh * n_kt;
        const unsigned grid = (unsigned)std::min<long long>(items, (long long)cus * per_cu);
        e = launch_kernel(kernel, dim3(grid), dim3(KV2_THREADS), stream, static_cast<const u16*>(p.q),
                          static_cast<const u16*>(p.k), static_cast<const u16*>(p.v),
                          static_cast<const u16*>(p.dout), p.lse, static_cast<const float*>(p.dsum),
                          p.dk, p.dv, p.nq, p.nk, p.bh, n_kt, c, p.scale);
    }
    return e;
}

template <int D>
hipError_t launch_d(const BwdProblem& p, hipStream_t stream) {
    if (p.causal)
        return p.grad_bf16 ? launch<D, true, true>(p, stream) : launch<D, true, false>(p, stream);
    return p.grad_bf16 ? launch<D, false, true>(p, stream) : launch<D, false, false>(p, stream);
}

}  // namespace

hipError_t launch_bwd(const BwdProblem& p, hipStream_t stream) {
    if (p.d == 64) return launch_d<64>(p, stream);
    if (p.d == 128) return launch_d<128>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
