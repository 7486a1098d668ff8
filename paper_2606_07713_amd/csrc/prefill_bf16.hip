// Fused attention prefill for bf16 inputs on gfx950 matrix cores.
//
// One workgroup owns one (batch*head, 256-query tile) and runs 8 waves of 32
// queries each.  The Q tile stays in registers for the whole key loop, K and V
// stream through LDS in 64-key tiles, and nothing but the output (and the
// optional LSE) is ever written to device memory: scores, exponentials and the
// running softmax statistics live in registers only (the DNF of eqs. dnf_attn
// and output_dnf: no K^T buffer, no score matrix, no softmax temporary).
//
// Orientation.  Each wave computes the transposed score tile S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16: K rows are the A operand, read in their stored
// order, so no K^T is ever formed (eq. mm_psi reads K by row).  In the
// accumulator layout a lane holds scores of ONE query (column = lane % 32) for
// 16 keys and lane l ^ 32 holds the other 16 keys of the same query, so the
// row max (Step I) and row sum (Step III) are in-lane reductions plus one
// v_permlane32_swap.  The output is accumulated transposed as well,
// O^T += V^T P^T: the P^T operand is the score accumulator converted to bf16
// in place, and the V^T operand is read from the row-major V tile with
// ds_read_b64_tr_b16 (a transposing LDS read), so V is never transposed either.
//
// Data movement.  K and V tiles go from device memory straight into LDS
// (buffer_load ... lds, 16 bytes per lane, no register staging) through
// two-stage rings; rows past Nk come back as zeros from the buffer bounds.
// LDS rows are stored with a 16-byte-chunk XOR swizzle instead of padding,
// because direct-to-LDS writes are contiguous per instruction.  The output
// (and, in the key-split layout, the Q tile) also passes through LDS, so that
// device memory is written (read) in whole rows rather than in the 8- or
// 16-byte pieces per row that the MFMA register layouts hold.
//
// Ping-pong.  Waves w and w + 4 share a SIMD.  The workgroup advances in
// phases separated by barriers; in each phase one group of four waves issues
// the matrix products of a tile (P(t-1) V(t-1) and S(t) = K(t) Q^T) while the
// other group runs the softmax of its previous tile on the vector ALU, and the
// groups swap roles every phase.  This keeps the matrix cores and the vector
// ALU of every SIMD busy at the same time.
//
// Softmax.  Scores are kept in raw units; with c = scale * log2(e) the weight
// of key j is 2^(s_j c - m) where m is a running reference (log2 units) in
// place of the row maximum.  A tile's weights are first formed against the
// current reference without computing the tile max; only when their partial
// sum exceeds kFastSumLimit (or overflows) is the reference raised, to
// kRefHeadroom above the tile max (and O, l rescaled), and the tile redone.
// The final O = acc / l uses the same reference for numerator and
// denominator, so any reference gives the same quotient: the softmax of
// Steps I-IV regrouped over key tiles.
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "prefill_bf16_common.h"

namespace moa {
namespace {

using namespace pf;

constexpr int BM = WAVES * 32;   // queries per workgroup (ping-pong layout)

__device__ __forceinline__ void wait_loads_to_lds() {
    __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): this wave's LDS-bound loads have landed
}

// KSPLIT = false: ping-pong over one key range, 8 waves x 32 queries = 256
//   queries per workgroup.
// KSPLIT = true: 4 query blocks x 2 key halves = 128 queries per workgroup;
//   group g streams key tiles of its half through its own LDS rings (both
//   groups in the same phase), and group 1 hands its softmax state (m, l, O)
//   to group 0 through LDS at the end for an exact merge.  Used for grids
//   the ping-pong layout would leave partly idle (see use_key_split).
// PARTIAL = true (with KSPLIT): split-K across workgroups for grids smaller
//   still.  Work item = (batch*head, query tile, key split s of n_splits):
//   the item covers the s-th of n_splits equal shares of the query tile's
//   visible key tiles and, instead of O, writes its partial state -- the
//   reference m (log2 units), the denominator l and the un-normalised output
//   acc -- to Out = ws_acc [bh*Nq][n_splits][D] and LSE = ws_ml
//   [bh*Nq][n_splits][2]; launch_split_combine merges the splits.  A share
//   with no key visible to a row leaves (m, l, acc) = (-inf, 0, 0).
template <int D, bool CAUSAL, bool OUT_BF16, bool KSPLIT, bool STRIDED, bool PARTIAL = false>
__global__ __launch_bounds__(THREADS, 1) void prefill_bf16_kernel(
    const u16* __restrict__ Q, const u16* __restrict__ K, const u16* __restrict__ V,
    void* __restrict__ Out, float* __restrict__ LSE, int Nq, int Nk, int n_bh, int n_qtiles, float c,
    Layout L, int n_splits) {
    static_assert(!PARTIAL || KSPLIT, "split-K items use the key-split layout");
    const Addr<D, STRIDED> A{L, Nq, Nk};
    using C = Cfg<D>;
    constexpr uint32_t RB = C::ROW_BYTES;
    constexpr int NG = KSPLIT ? 2 : 1;                    // independent key streams
    constexpr int QB = KSPLIT ? WAVES / 2 : WAVES;        // query blocks of 32
    constexpr int BMQ = QB * 32;                          // queries per workgroup
    constexpr int LOADERS = WAVES / NG;                   // waves loading one stream
    constexpr int LPW = C::TILE_BYTES / (LOADERS * 1024); // 16-byte loads per lane per tile
    static_assert(C::TILE_BYTES % (LOADERS * 1024) == 0, "tile must split into wave loads");
    // One LDS array per ring stage (each holding one tile per stream): the
    // compiler tracks direct-to-LDS loads per underlying object, so reads of
    // one stage need not wait for loads still landing in another.
    __shared__ __attribute__((aligned(1024))) unsigned char k_st0[NG * C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char k_st1[NG * C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char v_st0[NG * C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char v_st1[NG * C::TILE_BYTES];
    // Key split: the item's Q tile, BMQ rows in the tiles' swizzled layout,
    // loaded whole rows at a time and read by the waves of both key streams
    // as their MFMA fragments.
    __shared__ __attribute__((aligned(1024))) unsigned char q_st[KSPLIT ? BMQ * C::ROW_BYTES : 16];
    auto k_stage = [&](auto tag) -> unsigned char* {
        if constexpr (decltype(tag)::value == 0) return k_st0; else return k_st1;
    };
    auto v_stage = [&](auto tag) -> unsigned char* {
        if constexpr (decltype(tag)::value == 0) return v_st0; else return v_st1;
    };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // Key split: the key half decides the buffer descriptors of the tile
    // loads, so it is made visibly wave-uniform (scalar registers; a per-lane
    // value there makes the compiler loop over the lanes around every load).
    // The ping-pong layout keeps its phase group per lane: its register
    // budget is tighter, and scalar copies of the group cost it spills.
    const int grp = KSPLIT ? __builtin_amdgcn_readfirstlane(wave >> 2) : wave >> 2;
    const int qw = KSPLIT ? (wave & 3) : wave;       // query block of this wave
    const int lw = KSPLIT ? (wave & 3) : wave;       // index among the waves loading its stream
    const uint32_t g_off = KSPLIT ? (uint32_t)grp * C::TILE_BYTES : 0u;   // stream's slot in a stage
    const int col = lane & 31;     // query within the wave's 32
    const int half = lane >> 5;    // which 8-element k group of the MFMA operands

    const int off = Nk - Nq;       // causal: key j visible to query i iff j <= i + off
    // A negative scale is folded into Q's sign (exact for bf16) so that the
    // softmax below always sees c > 0.  A zero (or denormal) scale becomes the
    // smallest normal float: every weight still rounds to exactly 1, and a
    // masked score (-inf) still gives weight 0 rather than -inf * 0 = NaN.
    const uint32_t qflip = (c < 0.0f) ? 0x80008000u : 0u;
    c = fmaxf(fabsf(c), 1.17549435e-38f);

    for (int item = 0;; ++item) {
    int bh, qt;
    if (!item_of(blockIdx.x, item, gridDim.x, n_bh, n_qtiles, CAUSAL, bh, qt)) break;
    int split = 0;                 // key share of a split-K item
    if constexpr (PARTIAL) {
        split = qt % n_splits;
        qt /= n_splits;
    }
    const int q0 = qt * BMQ;

    const u16* Qh = Q + A.q_head(bh);
    const u16* Kh = K + A.k_head(bh);
    const u16* Vh = V + A.v_head(bh);

    // ---- a1: Q fragment for this lane's query, all of d, kept in registers.
    // Ping-pong: loaded straight into the fragments.  Key split (both key
    // streams hold the same queries): the workgroup's BMQ query rows go to
    // LDS once, 16 bytes per lane and whole rows per load instruction,
    // together with the first key tile; each wave then reads its fragments
    // (the K operand's read pattern, conflict-free under the same swizzle).
    // 14.5 against 15.1-15.5 us on B4 H8 1K d = 64; the ping-pong layout ran
    // 2% slower that way.  Rows past Nq read as zeros (buffer bounds) and are
    // never stored.
    const int qrow = q0 + qw * 32 + col;
    bf16x8 qf[D / 16];
    if constexpr (!KSPLIT) {
        const uint32_t qrb = (uint32_t)A.qr() * 2u;
        const auto rq = make_rsrc(Qh, rows_extent(Nq, qrb, RB));
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
            qf[s] = __builtin_bit_cast(bf16x8, buffer_load16(rq, (uint32_t)qrow * qrb + s * 32 + half * 16));
    }
    auto issue_q_load = [&]() {
        if constexpr (KSPLIT) {
            constexpr int QL = BMQ * C::CHUNKS / (WAVES * 64);   // 16-byte loads per lane
            static_assert(BMQ * C::CHUNKS % (WAVES * 64) == 0, "Q tile must split into wave loads");
            const uint32_t qrb = (uint32_t)A.qr() * 2u;
            const auto rq = make_rsrc(Qh + (size_t)q0 * A.qr(), rows_extent(Nq - q0, qrb, RB));
#pragma unroll
            for (int i = 0; i < QL; ++i) {
                const int slot = (wave * QL + i) * 64 + lane;
                const int row = slot / C::CHUNKS, p = slot % C::CHUNKS;
                buffer_load16_to_lds(rq, q_st + (wave * QL + i) * 1024,
                                     (uint32_t)row * qrb + (uint32_t)((p ^ swz<D>(row)) * 16));
            }
        }
    };
    auto read_q = [&]() {
        if constexpr (KSPLIT) {
#pragma unroll
            for (int s = 0; s < D / 16; ++s)
                qf[s] = *reinterpret_cast<const bf16x8*>(
                    q_st + (uint32_t)(qw * 32 + col) * RB + (uint32_t)(((2 * s + half) ^ swz<D>(col)) * 16));
        }
    };
    // A negative scale flips Q's sign bits once the fragments have arrived
    // (ping-pong: after the first key tile's load has been issued, so the two
    // loads are in flight together; no flip: nothing waits for Q before the
    // first product).
    auto flip_q = [&]() {
        if (qflip == 0u) return;
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
            u32x4 w = __builtin_bit_cast(u32x4, qf[s]);
            w ^= qflip;
            qf[s] = __builtin_bit_cast(bf16x8, w);
        }
    };

    // Key tiles of this workgroup, of this wave's stream, and of this wave.
    int kv_end = Nk;
    if (CAUSAL) kv_end = min(Nk, q0 + BMQ + off);
    const int n_kt = (kv_end + BN - 1) / BN;
    int t_lo = 0, n_range = n_kt;                             // this item's key tiles
    if constexpr (PARTIAL) {
        const int share = (n_kt + n_splits - 1) / n_splits;
        t_lo = min(n_kt, split * share);
        n_range = min(n_kt, t_lo + share) - t_lo;
    }
    const int n_first = KSPLIT ? (n_range + 1) / 2 : n_range;   // tiles of stream 0
    const int g_start = t_lo + ((KSPLIT && grp == 1) ? n_first : 0);   // first global tile of the stream
    const int g_count = (KSPLIT && grp == 1) ? n_range - n_first : n_first;
    const int n_iter = n_first;                               // slots every wave walks through
    const int wave_q_first = q0 + qw * 32;
    int w_end = n_kt;                                         // global tiles this wave needs
    if (CAUSAL) w_end = min(n_kt, (wave_q_first + 31 + off) / BN + 1);
    const int n_w = max(0, min(g_start + g_count, w_end) - g_start);   // local count

    // ---- a2: direct-to-LDS tile loads.  Lane l of the i-th load of loader lw
    // fills slot S = (lw*LPW + i)*64 + l of its stream's tile, which holds
    // logical chunk (S % CHUNKS) ^ swz(row) of row S / CHUNKS.
    // The global offsets follow each tensor's row stride (kr, vr elements).
    const uint32_t krb = (uint32_t)A.kr() * 2u, vrb = (uint32_t)A.vr() * 2u;
    uint32_t ld_koff[LPW], ld_voff[LPW];
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
        const int slot = (lw * LPW + i) * 64 + lane;
        const int row = slot / C::CHUNKS, p = slot % C::CHUNKS;
        const uint32_t chunk = (uint32_t)((p ^ swz<D>(row)) * 16);
        ld_koff[i] = (uint32_t)row * krb + chunk;
        ld_voff[i] = (uint32_t)row * vrb + chunk;
    }
    // Loads the stream's local tile t of K or V into `stage` (only while
    // t < g_count).
    auto issue_tile_load = [&](bool is_k, int t, unsigned char* stage) {
        const int kbase = (g_start + t) * BN;
        const u16* head = is_k ? Kh : Vh;
        const int rs = is_k ? A.kr() : A.vr();
        const auto r = make_rsrc(head + (size_t)kbase * rs, rows_extent(Nk - kbase, (uint32_t)rs * 2u, RB));
#pragma unroll
        for (int i = 0; i < LPW; ++i)
            buffer_load16_to_lds(r, stage + g_off + (lw * LPW + i) * 1024, is_k ? ld_koff[i] : ld_voff[i]);
    };

    // Per-lane LDS addresses of the MFMA operand reads (stage, key block and
    // key chunk are added as immediates; the stream's slot is folded in).
    uint32_t kaddr[D / 16];          // K rows: row = col (+32 kb), chunk 2s + half
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
        kaddr[s] = g_off + (uint32_t)col * RB + (uint32_t)(((2 * s + half) ^ swz<D>(col)) * 16);
    uint32_t vaddr[D / 32][2];       // V rows for ds_read_b64_tr_b16 (lo / hi key quads)
    {
        const int g = lane >> 4, j = (lane >> 2) & 3, q = lane & 3;
#pragma unroll
        for (int b = 0; b < D / 32; ++b)
#pragma unroll
            for (int h8 = 0; h8 < 2; ++h8) {
                const int row = 4 * (g >> 1) + j + 8 * h8;
                const int dv = dv_of<D>(b, 16 * (g & 1) + 4 * q);
                vaddr[b][h8] = g_off + (uint32_t)row * RB +
                               (uint32_t)((((dv >> 3) ^ swz<D>(row)) * 16) + (dv & 7) * 2);
            }
    }
    f32x16 oacc[D / 32];
#pragma unroll
    for (int b = 0; b < D / 32; ++b) oacc[b] = f32x16{};
    f32x16 sacc[BN / 32];            // S^T of the current tile
    bf16x8 pbuf[BN / 16];            // bf16 P^T of the current tile
    float m_run = kNegInf;           // running reference max, log2 units (scores * c)
    float neg_m = 0.0f;              // -m_run, or 0 while m_run is -inf (no visible key yet)
    float l_run = 0.0f;              // partial denominator over this half-wave's keys
    float alpha_pend = 1.0f;         // rescale owed to oacc before the next P.V
    bool rescale_pend = false;

    // ---- a3: S^T(t) = K_t . Q^T from K stage B.
    auto s_mfma = [&](auto stage_tag) {
        const unsigned char* ks = k_stage(stage_tag);
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb) sacc[kb] = f32x16{};
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
#pragma unroll
            for (int kb = 0; kb < BN / 32; ++kb) {
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(ks + kaddr[s] + kb * 32 * RB);
                sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], sacc[kb], 0, 0, 0);
            }
    };

    // ---- a6: O^T += V^T . P^T from V stage B.  Chunk cc covers keys
    // 16cc + 4*half + {0..3} and 16cc + 8 + 4*half + {0..3}, which is both the
    // key order of pbuf (the S^T accumulator layout) and that of the two
    // transposing reads.
    auto pv_mfma = [&](auto stage_tag) {
        unsigned char* vs = v_stage(stage_tag);
#pragma unroll
        for (int cc = 0; cc < BN / 16; ++cc)
#pragma unroll
            for (int b = 0; b < D / 32; ++b) {
                const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4s*)(vs + vaddr[b][0] + cc * 16 * RB));
                const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4s*)(vs + vaddr[b][1] + cc * 16 * RB));
                const v4s both[2] = {lo, hi};
                oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, both), pbuf[cc], oacc[b], 0, 0, 0);
            }
    };

    // ---- a4 + a5: softmax of tile t from sacc into pbuf.
    //
    // Weights are p = 2^(s c - m) against the running reference m, rounded to
    // bf16 for the P.V product; the denominator sums exactly those rounded
    // weights (v_dot2_f32_bf16 against ones), so numerator and denominator use
    // the same p.  exp_pack() returns the tile's partial sum (this lane's 32
    // keys).  Masked scores are -inf and c > 0, so their weight is exactly 0.
    auto exp_pack = [&](float nm) {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
        float part[2] = {0.0f, 0.0f};
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                u32x4 w;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int i = g * 8 + 2 * j;
                    const float p0 = exp2_hw(__builtin_fmaf(sacc[kb][i], c, nm));
                    const float p1 = exp2_hw(__builtin_fmaf(sacc[kb][i + 1], c, nm));
                    const bf16x2 pp = {(__bf16)p0, (__bf16)p1};
                    w[j] = __builtin_bit_cast(uint32_t, pp);
                    part[j & 1] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, part[j & 1], false);
                }
                pbuf[kb * 2 + g] = __builtin_bit_cast(bf16x8, w);
            }
        return part[0] + part[1];
    };

    // Causal / ragged tiles: scores of keys this query must not see become
    // -inf in place.
    auto apply_mask = [&](int t) {
        const int kbase = (g_start + t) * BN;
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = kbase + kb * 32 + (i >> 2) * 8 + half * 4 + (i & 3);
                const bool masked = key >= Nk || (CAUSAL && key > qrow + off);
                if (masked) sacc[kb][i] = kNegInf;
            }
    };

    // Step I on the tile: its row max; the reference is raised (and l, O owe
    // the factor 2^(m_old - m_new)) only when the tile exceeds it by more than
    // kRescaleSlack.
    auto raise_reference = [&]() {
        // The empty asm keeps the max from being hoisted onto the fast path
        // (the scores do not change between the passes below).
        float mx = kNegInf;
        asm volatile("" : "+v"(mx));
#pragma unroll
        for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kb][i]);
        const float mt = half_max(mx) * c;
        if (wave_any(mt > m_run + kRescaleSlack)) {
            // A row may have seen no visible key yet (its reference is still
            // -inf): there is nothing to rescale, and 2^(-inf - -inf) must
            // not be formed.
            const float m_new = fmaxf(m_run, mt + kRefHeadroom);
            const float alpha = (m_run == kNegInf) ? 0.0f : exp2_hw(m_run - m_new);
            l_run *= alpha;
            alpha_pend = rescale_pend ? alpha_pend * alpha : alpha;
            rescale_pend = true;
            m_run = m_new;
            neg_m = (m_new == kNegInf) ? 0.0f : -m_new;
        }
    };

    auto tile_needs_mask = [&](int t) {
        const int kbase = (g_start + t) * BN;
        return (kbase + BN > Nk) || (CAUSAL && kbase + BN - 1 > wave_q_first + off);
    };

    // Softmax of tile t.  The weights are first taken against the current
    // reference without computing the tile max; only if a partial sum exceeds
    // kFastSumLimit (or overflowed) is the reference raised and the tile
    // redone.  Any reference gives the same quotient, so this is exact.  A
    // row that has seen no key yet starts from its tile max plus kRefHeadroom
    // instead (a guessed reference far above its scores would underflow every
    // weight); rows still without a visible key keep reference -inf and take
    // weights 2^(s c) (neg_m = 0), all their scores being -inf.  The redo is a
    // second straight-line pass; the fast path then carries no copies of the
    // softmax state (a two-pass loop made the compiler copy m, l and the
    // rescale factor at every tile).
    auto softmax_phase = [&](int t) {
        if (t >= n_w) return;
        if (tile_needs_mask(t)) apply_mask(t);
        if (wave_any(m_run == kNegInf)) raise_reference();
        float part = exp_pack(neg_m);
        if (wave_any(!(part <= kFastSumLimit))) {
            raise_reference();
            part = exp_pack(neg_m);
        }
        l_run += part;
    };

    // Matrix phase of tile t: P(t-1) V(t-1) then S(t).  K(t) sits in K stage
    // t & 1 and V(t-1) in V stage (t-1) & 1 = PAR ^ 1.
    auto gemm_phase = [&](int t, auto par_tag) {
        constexpr int P = decltype(par_tag)::value;
        if (rescale_pend) {
#pragma unroll
            for (int b = 0; b < D / 32; ++b) oacc[b] *= alpha_pend;
            rescale_pend = false;
        }
        if (t >= 1 && t - 1 < n_w) pv_mfma(std::integral_constant<int, 1 - P>{});
        if (t < n_w) s_mfma(std::integral_constant<int, P>{});
    };

    // Slots t = 0, 1, 2, ... over the stream's local tiles.  Ping-pong: the
    // leading group runs gemm(t) in the first half of slot t and softmax(t) in
    // the second; the trailing group runs softmax(t-1), then gemm(t).  Key
    // split: every wave leads.  K(t+1) and V(t) are loaded during slot t into
    // the stages freed by slot t - 1 and waited for at its end.  The barrier
    // between the two halves of a slot only swaps the groups' roles: it
    // guards no LDS data, so it carries no memory fence (which would wait for
    // the loads in flight at mid-slot).
    const bool lead = KSPLIT || grp == 0;
    issue_q_load();
    if (g_count > 0) issue_tile_load(true, 0, k_st0);
    if constexpr (!KSPLIT) flip_q();
    wait_loads_to_lds();
    __syncthreads();
    if constexpr (KSPLIT) {
        read_q();
        flip_q();
    }
    for (int t = 0; t <= n_iter; t += 2) {
        // ---- even tile t (parity 0)
        if (t + 1 < g_count) issue_tile_load(true, t + 1, k_st1);
        if (t < g_count) issue_tile_load(false, t, v_st0);
        if (lead) gemm_phase(t, S0{});
        else if (t >= 1) softmax_phase(t - 1);
        if constexpr (!KSPLIT) barrier_no_fence();
        if (lead) softmax_phase(t);
        else gemm_phase(t, S0{});
        wait_loads_to_lds();
        __syncthreads();
        if (t + 1 > n_iter) break;
        // ---- odd tile t + 1 (parity 1)
        if (t + 2 < g_count) issue_tile_load(true, t + 2, k_st0);
        if (t + 1 < g_count) issue_tile_load(false, t + 1, v_st1);
        if (lead) gemm_phase(t + 1, S1{});
        else softmax_phase(t);
        if constexpr (!KSPLIT) barrier_no_fence();
        if (lead) softmax_phase(t + 1);
        else gemm_phase(t + 1, S1{});
        wait_loads_to_lds();
        __syncthreads();
    }

    // Key split: group 1 hands (m, l, O^T) to group 0, which merges exactly:
    // M = max(m0, m1), O = 2^(m0-M) O0 + 2^(m1-M) O1, l likewise.  The K ring
    // holds the O^T blocks ([reg][lane], lane-contiguous), the V ring m and l.
    if constexpr (KSPLIT) {
        float* xo = reinterpret_cast<float*>((qw < 2 ? k_st0 : k_st1) +
                                             (qw & 1) * (D / 2) * 64 * sizeof(float));
        float* xml = reinterpret_cast<float*>(v_st0) + qw * 2 * 64;
        if (grp == 1) {
#pragma unroll
            for (int b = 0; b < D / 32; ++b)
#pragma unroll
                for (int i = 0; i < 16; ++i) xo[(b * 16 + i) * 64 + lane] = oacc[b][i];
            xml[lane] = m_run;
            xml[64 + lane] = l_run;
        }
        __syncthreads();
        if (grp == 0) {
        const float m1 = xml[lane], l1 = xml[64 + lane];
        const float mm = fmaxf(m_run, m1);
        const float a0 = (m_run == kNegInf) ? 0.0f : exp2_hw(m_run - mm);
        const float a1 = (m1 == kNegInf) ? 0.0f : exp2_hw(m1 - mm);
        l_run = l_run * a0 + l1 * a1;
#pragma unroll
        for (int b = 0; b < D / 32; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[b][i] = oacc[b][i] * a0 + xo[(b * 16 + i) * 64 + lane] * a1;
        m_run = mm;
        }
    }

    // ---- Output rows.  In the O^T accumulator layout a lane holds pieces of
    // one query row, so a direct store would write 32 rows per instruction.
    // A wave first puts its 32 rows into LDS in row order (16-byte chunks
    // XOR-swizzled by row), then stores whole rows, 16 bytes per lane.  Its
    // staging area (32 rows of 2*D bytes) is a slice of the tile stages that
    // no wave reads any more: the ping-pong layout's four stages hold two
    // waves each; in the key split each wave of group 0 reuses the area it
    // read its partner's state from.  The lane index goes through an empty
    // asm so that the staging addresses are formed here: hoisted out of the
    // item loop they would hold ~24 registers through the key loop and cost
    // its LDS read-ahead.
    unsigned char* stg;
    if constexpr (KSPLIT) {
        stg = (qw < 2 ? k_st0 : k_st1) + (qw & 1) * (D / 2) * 64 * sizeof(float);
    } else {
        unsigned char* st = (qw < 2) ? k_st0 : (qw < 4) ? k_st1 : (qw < 6) ? v_st0 : v_st1;
        stg = st + (qw & 1) * 32 * RB;
    }
    // fp32 rows (the split-K partial state or fp32 O), times `scl`, in two
    // passes of D/2 columns: row_ptr(r) is the destination of row r of the
    // wave's 32, or null for rows past Nq.
    auto store_rows_f32 = [&](float scl, auto row_ptr) {
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int cl = ln & 31, hf = ln >> 5;
        constexpr int HB = D * 2;       // bytes of a half row (D/2 floats)
        constexpr int HCH = HB / 16;    // its 16-byte chunks
        constexpr int RPI = 64 / HCH;   // rows per store instruction
        const int rr = ln / HCH, ch = ln % HCH;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int b = 0; b < D / 32; ++b)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    if (dv_of<D>(b, g * 8) / (D / 2) != h) continue;
                    const int c = (dv_of<D>(b, g * 8 + hf * 4) - h * (D / 2)) / 4;
                    *reinterpret_cast<float4*>(stg + (uint32_t)cl * HB +
                                               (uint32_t)((c ^ (cl & (HCH - 1))) * 16)) =
                        make_float4(oacc[b][g * 4 + 0] * scl, oacc[b][g * 4 + 1] * scl,
                                    oacc[b][g * 4 + 2] * scl, oacc[b][g * 4 + 3] * scl);
                }
            wait_lgkmcnt0();   // this wave's rows are in LDS (only this wave reads them)
#pragma unroll
            for (int i = 0; i < 32 / RPI; ++i) {
                const int r = i * RPI + rr;
                const float4 v = *reinterpret_cast<const float4*>(
                    stg + (uint32_t)r * HB + (uint32_t)((ch ^ (r & (HCH - 1))) * 16));
                float* dst = row_ptr(r);
                if (dst != nullptr) *reinterpret_cast<float4*>(dst + h * (D / 2) + ch * 4) = v;
            }
        }
    };

    // ---- a8 (split-K): the partial state of this key share, un-normalised,
    // for the combine pass.
    if constexpr (PARTIAL) {
    if (grp == 0) {
        const float l_tot = half_sum(l_run);
        store_rows_f32(1.0f, [&](int r) -> float* {
            const int q = wave_q_first + r;
            return q < Nq ? static_cast<float*>(Out) + (((size_t)bh * Nq + q) * n_splits + split) * D
                          : nullptr;
        });
        if (qrow < Nq && half == 0) {
            const size_t prow = ((size_t)bh * Nq + qrow) * n_splits + split;
            LSE[prow * 2 + 0] = m_run;
            LSE[prow * 2 + 1] = l_tot;
        }
    }
    } else {
    // ---- a7: epilogue, O = acc / l: the only device-memory write (key
    // split: by group 0, which holds the merged state).
    if (!KSPLIT || grp == 0) {
    const float l_tot = half_sum(l_run);
    const float inv = 1.0f / l_tot;
    if constexpr (OUT_BF16) {
        constexpr int CHK = C::CHUNKS;
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int cl = ln & 31, hf = ln >> 5;
#pragma unroll
        for (int b = 0; b < D / 32; ++b)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int dv = dv_of<D>(b, g * 8 + hf * 4);
                const uint2 w = make_uint2(pack_bf16x2(oacc[b][g * 4 + 0] * inv, oacc[b][g * 4 + 1] * inv),
                                           pack_bf16x2(oacc[b][g * 4 + 2] * inv, oacc[b][g * 4 + 3] * inv));
                const uint32_t a = (uint32_t)cl * RB +
                                   (uint32_t)((((dv >> 3) ^ (cl & (CHK - 1))) * 16) + (dv & 7) * 2);
                *reinterpret_cast<uint2*>(stg + a) = w;
            }
        wait_lgkmcnt0();   // this wave's rows are in LDS (only this wave reads them)
        constexpr int RPI = 64 / CHK;   // rows per store instruction
        const int rr = ln / CHK, ch = ln % CHK;
#pragma unroll
        for (int i = 0; i < 32 / RPI; ++i) {
            const int r = i * RPI + rr;
            const uint4 v = *reinterpret_cast<const uint4*>(
                stg + (uint32_t)r * RB + (uint32_t)((ch ^ (r & (CHK - 1))) * 16));
            const int q = wave_q_first + r;
            if (q < Nq)
                *reinterpret_cast<uint4*>(static_cast<u16*>(Out) + (size_t)A.o_head(bh) +
                                          (size_t)q * A.orow() + ch * 8) = v;
        }
    } else {
        store_rows_f32(inv, [&](int r) -> float* {
            const int q = wave_q_first + r;
            return q < Nq ? static_cast<float*>(Out) + (size_t)A.o_head(bh) + (size_t)q * A.orow()
                          : nullptr;
        });
    }
    if (LSE != nullptr && half == 0 && qrow < Nq)
        LSE[(size_t)bh * Nq + qrow] = (m_run + __log2f(l_tot)) * kLn2;
    }
    }
    // Every wave is done with this item's LDS before the next item's first
    // tile loads land there: its LDS reads have returned (their values are
    // consumed above; the wait makes it explicit), and the barrier orders
    // them before any wave's next loads.  No memory fence: it would wait for
    // the O stores just issued (vmcnt counts stores too), which nothing in
    // this workgroup reads.
    wait_lgkmcnt0();
    barrier_no_fence();
    }
}

// Layout choice.  Work items are 256-query tiles (ping-pong) or 128-query
// tiles (key split: two key streams per workgroup and an exact merge, which
// doubles the items of a grid).  With the causal mask the snake deal balances
// unequal items, and the ping-pong layout is the faster one from one item per
// compute unit on (e.g. B1 H80 1K d = 128: 37.9 against 46.1 us).  Without it
// every item costs the same, so a grid runs in whole rounds of items per
// compute unit.  The key split halves the rounds of a grid smaller than the
// GPU (B4 H8 1K d = 64: 17.2 against 24.9 us), and evens out grids of one to
// two items per compute unit when its half-size items need at most three
// quarters of the ping-pong's rounds and every key stream gets at least 512
// keys (B1 H80 1K: 66.8 against 71.8 us at d = 128, 39.5 against 44.4 at
// d = 64; with 700 keys the ping-pong layout stays ahead, 56.2 against 58.0
// us on B1 H128 600 x 700).  Otherwise the ping-pong layout (B1 H48 1K
// d = 128: 40.7 against 47.9 us; B1 H128 1K: 79.5 against 89.9).
template <bool CAUSAL>
bool use_key_split(long long items_pp, long long items_ks, int nk, int cus) {
    if (items_pp < cus) return true;
    if (CAUSAL || nk < 1024) return false;
    const long long rounds_pp2 = 2 * ((items_pp + cus - 1) / cus);   // in key-split item units
    const long long rounds_ks2 = (items_ks + cus - 1) / cus;
    return 4 * rounds_ks2 <= 3 * rounds_pp2;
}

// One persistent launch: as many workgroups as the device holds at once, at
// most one per work item.  `n_qtiles` counts query tiles times key splits;
// `out` and `lse` are O and LSE, or the two partial-state arrays (PARTIAL).
template <int D, bool CAUSAL, bool OUT_BF16, bool KSPLIT, bool STRIDED, bool PARTIAL = false>
hipError_t launch_persistent(const Problem& p, int n_qtiles, float c, void* out, float* lse,
                             int n_splits, hipStream_t stream) {
    auto kernel = prefill_bf16_kernel<D, CAUSAL, OUT_BF16, KSPLIT, STRIDED, PARTIAL>;
    static const int per_cu = [&] {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, THREADS, 0) != hipSuccess) n = 1;
        return n > 0 ? n : 1;
    }();
    int cus = 0;
    const hipError_t e = device_cus(stream, cus);
    if (e != hipSuccess) return e;
    const long long items = (long long)p.bh * n_qtiles;
    const unsigned grid = (unsigned)std::min<long long>(items, (long long)cus * per_cu);
    return launch_kernel(kernel, dim3(grid), dim3(THREADS), stream,
                         static_cast<const u16*>(p.q), static_cast<const u16*>(p.k),
                         static_cast<const u16*>(p.v), out, lse, p.nq, p.nk, p.bh, n_qtiles, c,
                         p.lay, n_splits);
}

template <int D, bool CAUSAL, bool OUT_BF16, bool STRIDED>
hipError_t launch(const Problem& p, hipStream_t stream) {
    const float c = p.scale * kLog2e;
    const int qt_pp = (p.nq + BM - 1) / BM;
    const int qt_ks = (p.nq + BM / 2 - 1) / (BM / 2);
    if (p.splits > 1) {
        // Split-K: partial states of every key share, then the exact merge.
        float* ws_acc = p.ws;
        float* ws_ml = p.ws + (size_t)p.bh * p.nq * p.splits * D;
        const hipError_t e = launch_persistent<D, CAUSAL, false, true, STRIDED, true>(
            p, qt_ks * p.splits, c, ws_acc, ws_ml, p.splits, stream);
        if (e != hipSuccess) return e;
        return launch_split_combine(p, p.splits, ws_acc, ws_ml, stream);
    }
    int cus = 0;
    const hipError_t e = device_cus(stream, cus);
    if (e != hipSuccess) return e;
    if (p.nk > BN &&
        use_key_split<CAUSAL>((long long)p.bh * qt_pp, (long long)p.bh * qt_ks, p.nk, cus))
        return launch_persistent<D, CAUSAL, OUT_BF16, true, STRIDED>(p, qt_ks, c, p.o, p.lse, 1,
                                                                     stream);
    return launch_persistent<D, CAUSAL, OUT_BF16, false, STRIDED>(p, qt_pp, c, p.o, p.lse, 1, stream);
}

template <int D, bool STRIDED>
hipError_t launch_s(const Problem& p, hipStream_t stream) {
    if (p.causal)
        return p.out_bf16 ? launch<D, true, true, STRIDED>(p, stream)
                          : launch<D, true, false, STRIDED>(p, stream);
    return p.out_bf16 ? launch<D, false, true, STRIDED>(p, stream)
                      : launch<D, false, false, STRIDED>(p, stream);
}

template <int D>
hipError_t launch_d(const Problem& p, hipStream_t stream) {
    return is_contiguous(p) ? launch_s<D, false>(p, stream) : launch_s<D, true>(p, stream);
}

}  // namespace

static_assert(BM == kPrefillBf16RowsPerBlock, "row tile mismatch");

hipError_t launch_prefill_bf16(const Problem& p, hipStream_t stream) {
    if (p.d == 64) return launch_d<64>(p, stream);
    if (p.d == 128) return launch_d<128>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
