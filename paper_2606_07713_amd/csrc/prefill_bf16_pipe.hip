// Fused attention prefill for bf16 inputs on gfx950 matrix cores: per-wave
// software pipeline.
//
// A work item is one (batch*head, 256-query tile); a workgroup of 8 waves
// walks its items persistently and each wave owns 32 queries.  The Q tile
// stays in registers, K and V stream through LDS, and only O (and the
// optional LSE) is written to device memory: scores, weights and the running
// softmax statistics stay in registers (the DNF of eqs. dnf_attn and
// output_dnf; no K^T, no score matrix).
//
// Orientation (as in the ping-pong kernel): S^T = K Q^T with K rows as the
// MFMA A operand read in stored order, so a lane holds the scores of ONE
// query (16 keys; lane ^ 32 the other 16), and O^T += V^T P^T with P^T taken
// from the score accumulator packed to bf16 and V^T read by transposing LDS
// reads (ds_read_b64_tr_b16).
//
// Pipeline.  Keys advance in steps of 32.  In step t every wave issues, in
// one straight-line block, the matrix products S(t+1) = K(t+1) Q^T and
// O^T += V(t-1)^T P(t-1)^T together with the softmax of step t (vector ALU
// and exp), so each wave keeps the matrix cores and the vector ALU busy at
// once; two waves per SIMD interleave further.  There is no phase barrier
// between waves.
//
// Data movement.  K and V stages of 64 keys go from device memory into
// registers (16 bytes per lane, coalesced; rows past Nk read as zeros through
// the buffer bound) one stage iteration before they are stored into a
// two-stage LDS ring, so a load has a whole iteration to arrive and the
// compiler tracks it like any register load.  One barrier per 64 keys, without
// the memory-model fences of __syncthreads(), publishes a stage and frees the
// other.
//
// Softmax.  Scores stay in raw units; with c = scale * log2(e) the weight of
// key j is 2^(s_j c - m) for a running reference m (log2 units) that is
// raised, with O and l rescaled, only when a step exceeds it by more than
// kRescaleSlack.  The fast step takes the weights against the current
// reference without the step max and only checks the partial sum.
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "prefill_bf16_common.h"

namespace moa {
namespace {

using namespace pf;

constexpr int BMQ = WAVES * 32;  // queries per work item
constexpr int SUB = 32;          // keys per pipeline step (one S^T accumulator)
constexpr int RING = 2;          // LDS stages per K ring and per V ring

template <int N>
using Tag = std::integral_constant<int, N>;

template <int D, bool CAUSAL, bool OUT_BF16, bool STRIDED>
__global__ __launch_bounds__(THREADS, 1) void prefill_pipe_kernel(
    const u16* __restrict__ Q, const u16* __restrict__ K, const u16* __restrict__ V,
    void* __restrict__ Out, float* __restrict__ LSE, int Nq, int Nk, int n_bh, int n_qtiles, float c,
    Layout L) {
    const Addr<D, STRIDED> A{L, Nq, Nk};
    using C = Cfg<D>;
    constexpr uint32_t RB = C::ROW_BYTES;
    constexpr int LPS = C::TILE_BYTES / (WAVES * 1024);   // 16-byte loads per lane per stage
    static_assert(C::TILE_BYTES % (WAVES * 1024) == 0, "a stage must split into wave loads");
    __shared__ __attribute__((aligned(1024))) unsigned char k_r0[C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char k_r1[C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char v_r0[C::TILE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char v_r1[C::TILE_BYTES];
    auto kslot = [&](auto tag) __attribute__((always_inline)) -> unsigned char* {
        if constexpr (decltype(tag)::value % RING == 0) return k_r0;
        else return k_r1;
    };
    auto vslot = [&](auto tag) __attribute__((always_inline)) -> unsigned char* {
        if constexpr (decltype(tag)::value % RING == 0) return v_r0;
        else return v_r1;
    };

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int col = lane & 31;     // query within the wave's 32
    const int half = lane >> 5;    // which 8-element k group of the MFMA operands
    const int off = Nk - Nq;       // causal: key j visible to query i iff j <= i + off

    // A negative scale is folded into Q's sign (exact for bf16) so that the
    // softmax always sees c > 0.  A zero (or denormal) scale becomes the
    // smallest normal float: every weight still rounds to exactly 1, and a
    // masked score (-inf) still gives weight 0 rather than -inf * 0 = NaN.
    const uint32_t qflip = (c < 0.0f) ? 0x80008000u : 0u;
    c = fmaxf(fabsf(c), 1.17549435e-38f);

    // Stage loads: the i-th 16-byte load of lane l of wave w reads chunk
    // S = (w*LPS + i)*64 + l of the stage (contiguous across the workgroup)
    // and stores it at LDS row S / CHUNKS, physical chunk (S % CHUNKS) ^
    // swz(row).
    // The global offsets follow each tensor's row stride (kr, vr elements).
    const uint32_t krb = (uint32_t)A.kr() * 2u, vrb = (uint32_t)A.vr() * 2u;
    uint32_t st_woff[LPS], st_koff[LPS], st_voff[LPS];
#pragma unroll
    for (int i = 0; i < LPS; ++i) {
        const int slot = (wave * LPS + i) * 64 + lane;
        const int row = slot / C::CHUNKS, p = slot % C::CHUNKS;
        st_woff[i] = (uint32_t)row * RB + (uint32_t)((p ^ swz<D>(row)) * 16);
        st_koff[i] = (uint32_t)row * krb + (uint32_t)(p * 16);
        st_voff[i] = (uint32_t)row * vrb + (uint32_t)(p * 16);
    }
    // Per-lane LDS addresses of the MFMA operand reads; the 32-key half of a
    // stage and the 16-key chunk are added as immediates.
    uint32_t kaddr[D / 16];          // K rows: row = col (+32 u), chunk 2s + half
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
        kaddr[s] = (uint32_t)col * RB + (uint32_t)(((2 * s + half) ^ swz<D>(col)) * 16);
    uint32_t vaddr[D / 32][2];       // V rows for ds_read_b64_tr_b16 (lo / hi key quads)
    {
        const int g = lane >> 4, j = (lane >> 2) & 3, q = lane & 3;
#pragma unroll
        for (int b = 0; b < D / 32; ++b)
#pragma unroll
            for (int h8 = 0; h8 < 2; ++h8) {
                const int row = 4 * (g >> 1) + j + 8 * h8;
                const int dv = dv_of<D>(b, 16 * (g & 1) + 4 * q);
                vaddr[b][h8] = (uint32_t)row * RB +
                               (uint32_t)((((dv >> 3) ^ swz<D>(row)) * 16) + (dv & 7) * 2);
            }
    }

    for (int item = 0;; ++item) {
        int bh, qt;
        if (!item_of(blockIdx.x, item, gridDim.x, n_bh, n_qtiles, CAUSAL, bh, qt)) break;
        const int q0 = qt * BMQ;
        const u16* Qh = Q + A.q_head(bh);
        const u16* Kh = K + A.k_head(bh);
        const u16* Vh = V + A.v_head(bh);

        // ---- a1: Q fragment for this lane's query, all of d, in registers.
        // Rows past Nq read as zeros (buffer bounds) and are never stored.
        const int qrow = q0 + wave * 32 + col;
        bf16x8 qf[D / 16];
        {
            const uint32_t qrb = (uint32_t)A.qr() * 2u;
            const auto rq = make_rsrc(Qh, rows_extent(Nq, qrb, RB));
#pragma unroll
            for (int s = 0; s < D / 16; ++s)
                qf[s] = __builtin_bit_cast(bf16x8,
                                           buffer_load16(rq, (uint32_t)qrow * qrb + s * 32 + half * 16));
        }
        // A negative scale flips Q's sign bits once the fragments have
        // arrived, after the first stage loads are issued (no flip: nothing
        // waits for Q before the first product).
        auto flip_q = [&]() __attribute__((always_inline)) {
            if (qflip == 0u) return;
#pragma unroll
            for (int s = 0; s < D / 16; ++s) {
                u32x4 w = __builtin_bit_cast(u32x4, qf[s]);
                w ^= qflip;
                qf[s] = __builtin_bit_cast(bf16x8, w);
            }
        };

        // Steps of the item (over all its waves) and of this wave.
        const int kv_end = CAUSAL ? min(Nk, q0 + BMQ + off) : Nk;
        const int n_sub = (kv_end + SUB - 1) / SUB;
        const int n_iters = (n_sub + 1) / 2;       // stage iterations of two steps
        const int wave_q_first = q0 + wave * 32;
        int n_w = n_sub;
        if (wave_q_first >= Nq) n_w = 0;
        else if (CAUSAL) n_w = min(n_sub, (wave_q_first + 31 + off) / SUB + 1);

        // ---- a2: stage j (keys 64j .. 64j + 63) of K or V: this lane's
        // share into registers (rows past Nk read as zeros), then into an LDS
        // slot one stage iteration later.
        auto load_stage = [&](bool is_k, int j, uint4 (&st)[LPS]) __attribute__((always_inline)) {
            const int kb = min(j * BN, Nk);
            const u16* head = is_k ? Kh : Vh;
            const int rs = is_k ? A.kr() : A.vr();
            const auto r = make_rsrc(head + (size_t)kb * rs, rows_extent(Nk - kb, (uint32_t)rs * 2u, RB));
#pragma unroll
            for (int i = 0; i < LPS; ++i) st[i] = buffer_load16(r, is_k ? st_koff[i] : st_voff[i]);
        };
        auto store_stage = [&](unsigned char* slot, const uint4 (&st)[LPS]) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < LPS; ++i) *reinterpret_cast<uint4*>(slot + st_woff[i]) = st[i];
        };
        uint4 stK[LPS], stV[LPS];        // stages in flight: K(i + 3), V(i + 2)

        f32x16 oacc[D / 32];
#pragma unroll
        for (int b = 0; b < D / 32; ++b) oacc[b] = f32x16{};
        f32x16 sA, sB;                   // S^T of even / odd steps
        bf16x8 pA[2], pB[2];             // bf16 P^T of even / odd steps
        float m_run = kNegInf;           // running reference, log2 units (scores * c)
        float l_run = 0.0f;              // partial denominator over this half-wave's keys
        float alpha_pend = 1.0f;         // rescale owed to oacc before the next P.V
        bool rescale_pend = false;

        // ---- a3: S^T = K Q^T for the 32 keys of half u of a K stage.
        auto s_mfma = [&](const unsigned char* ks, int u, f32x16& acc) __attribute__((always_inline)) {
            acc = f32x16{};
#pragma unroll
            for (int s = 0; s < D / 16; ++s) {
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(ks + kaddr[s] + u * 32 * RB);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], acc, 0, 0, 0);
            }
        };

        // ---- a6: O^T += V^T P^T for half u of a V stage.  Chunk cc covers
        // keys 16cc + 4*half + {0..3} and 16cc + 8 + 4*half + {0..3}: the key
        // order of the S^T accumulator and of the two transposing reads.
        auto pv_mfma = [&](const unsigned char* vs, int u, const bf16x8 (&pb)[2]) __attribute__((always_inline)) {
#pragma unroll
            for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
                for (int b = 0; b < D / 32; ++b) {
                    const int cc = 2 * u + c2;
                    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (lds_v4s*)(vs + vaddr[b][0] + cc * 16 * RB));
                    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (lds_v4s*)(vs + vaddr[b][1] + cc * 16 * RB));
                    const v4s both[2] = {lo, hi};
                    oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, both), pb[c2], oacc[b], 0, 0, 0);
                }
        };

        // ---- a4 + a5: weights of a step, p = 2^(s c - m), rounded to bf16
        // in pairs; the denominator sums exactly those rounded weights
        // (v_dot2_f32_bf16 against ones).  Returns this lane's partial sum
        // over its 16 keys.  Masked scores are -inf and c > 0: weight 0.
        auto exp_pack = [&](const f32x16& s, bf16x8 (&pb)[2], float neg_m) __attribute__((always_inline)) {
            typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
            const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
            float part[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                u32x4 w;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int i = g * 8 + 2 * j;
                    const float p0 = exp2_hw(__builtin_fmaf(s[i], c, neg_m));
                    const float p1 = exp2_hw(__builtin_fmaf(s[i + 1], c, neg_m));
                    const bf16x2 pp = {(__bf16)p0, (__bf16)p1};
                    w[j] = __builtin_bit_cast(uint32_t, pp);
                    part[j] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, part[j], false);
                }
                pb[g] = __builtin_bit_cast(bf16x8, w);
            }
            return (part[0] + part[1]) + (part[2] + part[3]);
        };

        // Causal / ragged steps: scores of keys this query must not see
        // become -inf in place.
        auto apply_mask = [&](f32x16& s, int t) __attribute__((always_inline)) {
            const int kbase = t * SUB;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = kbase + (i >> 2) * 8 + half * 4 + (i & 3);
                const bool masked = key >= Nk || (CAUSAL && key > qrow + off);
                if (masked) s[i] = kNegInf;
            }
        };
        auto step_needs_mask = [&](int t) __attribute__((always_inline)) {
            const int kbase = t * SUB;
            return (kbase + SUB > Nk) || (CAUSAL && kbase + SUB - 1 > wave_q_first + off);
        };

        // Step I on a step's scores: the row max; the reference is raised
        // (l now, O before its next P.V) only when the step exceeds it by
        // more than kRescaleSlack.  A row that has seen no visible key yet
        // (reference -inf) has nothing to rescale.
        auto raise_reference = [&](const f32x16& s) __attribute__((always_inline)) {
            // The empty asm keeps the max from being hoisted onto the fast
            // path.
            float mx = kNegInf;
            asm volatile("" : "+v"(mx));
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[i]);
            const float mt = half_max(mx) * c;
            if (wave_any(mt > m_run + kRescaleSlack)) {
                const float m_new = fmaxf(m_run, mt + kRefHeadroom);
                const float alpha = (m_run == kNegInf) ? 0.0f : exp2_hw(m_run - m_new);
                l_run *= alpha;
                alpha_pend = rescale_pend ? alpha_pend * alpha : alpha;
                rescale_pend = true;
                m_run = m_new;
            }
        };
        auto apply_rescale = [&]() __attribute__((always_inline)) {
#pragma unroll
            for (int b = 0; b < D / 32; ++b) oacc[b] *= alpha_pend;
            rescale_pend = false;
        };

        // Softmax of step t: weights against the current reference without
        // the step max; only if a partial sum exceeds kFastSumLimit (or
        // overflowed) is the reference raised and the step redone.  Any
        // reference gives the same quotient, so this is exact.  A row that
        // has seen no key yet starts from its step max plus kRefHeadroom
        // instead (a guessed reference far above its scores would underflow
        // every weight); rows
        // still without a visible key take reference 0, all their scores
        // being -inf.
        auto softmax_pre = [&](f32x16& s, int t) __attribute__((always_inline)) {
            if (step_needs_mask(t)) apply_mask(s, t);
            if (wave_any(m_run == kNegInf)) raise_reference(s);
        };
        auto softmax_post = [&](const f32x16& s, bf16x8 (&pb)[2], float part) __attribute__((always_inline)) {
            if (wave_any(!(part <= kFastSumLimit))) {
                raise_reference(s);
                part = exp_pack(s, pb, m_run == kNegInf ? 0.0f : -m_run);
            }
            l_run += part;
        };

        // The three parts of a full step written as one interleaved sequence:
        // the NOPS MFMA operands are read two MFMAs ahead of use (the K rows
        // of S(t+1), then the V^T chunks of P.V(t-1)), and the softmax of
        // step t is cut into 16 pieces (half a weight pair each) spread over
        // the MFMAs, so that every wave issues matrix, LDS and vector work
        // side by side.  (The compiler may reorder within the block; pinning
        // this order with scheduling barriers measured slower.)
        auto fused_step = [&](const unsigned char* ks, int ku, const unsigned char* vs, int vu,
                              f32x16& s_next, const f32x16& s_cur, bf16x8 (&p_cur)[2],
                              const bf16x8 (&p_prev)[2]) __attribute__((always_inline)) {
            constexpr int NK = D / 16;             // K operands: S(t+1) k-steps
            constexpr int NOPS = 2 * NK;           // plus V^T operands: 2 chunks x D/32 blocks
            constexpr int PIECES = 16;             // softmax pieces
            typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
            const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
            const float neg_m = m_run == kNegInf ? 0.0f : -m_run;
            auto read_op = [&](int j) __attribute__((always_inline)) -> bf16x8 {
                if (j < NK)
                    return *reinterpret_cast<const bf16x8*>(ks + kaddr[j] + ku * 32 * RB);
                const int c2 = (j - NK) / (D / 32), b = (j - NK) % (D / 32);
                const int cc = 2 * vu + c2;
                const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4s*)(vs + vaddr[b][0] + cc * 16 * RB));
                const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4s*)(vs + vaddr[b][1] + cc * 16 * RB));
                const v4s both[2] = {lo, hi};
                return __builtin_bit_cast(bf16x8, both);
            };
            float pe[16];                          // weights of the step, fp32
            uint32_t wd[8];                        // ... as bf16 pairs
            float part[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            // Piece q: pair r = q / 2 of scores (2r, 2r + 1); the first half
            // forms both weights, the second rounds the pair and adds it.
            auto piece = [&](int q) __attribute__((always_inline)) {
                const int r = q >> 1;
                if ((q & 1) == 0) {
                    pe[2 * r] = exp2_hw(__builtin_fmaf(s_cur[2 * r], c, neg_m));
                    pe[2 * r + 1] = exp2_hw(__builtin_fmaf(s_cur[2 * r + 1], c, neg_m));
                } else {
                    const bf16x2 pp = {(__bf16)pe[2 * r], (__bf16)pe[2 * r + 1]};
                    wd[r] = __builtin_bit_cast(uint32_t, pp);
                    part[r & 3] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, part[r & 3], false);
                }
            };
            bf16x8 ops[NOPS];
            ops[0] = read_op(0);
            ops[1] = read_op(1);
            s_next = f32x16{};
#pragma unroll
            for (int j = 0; j < NOPS; ++j) {
                if (j + 2 < NOPS) ops[j + 2] = read_op(j + 2);
                if (j < NK) {
                    s_next = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ops[j], qf[j], s_next, 0, 0, 0);
                } else {
                    const int c2 = (j - NK) / (D / 32), b = (j - NK) % (D / 32);
                    oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ops[j], p_prev[c2], oacc[b],
                                                                      0, 0, 0);
                }
#pragma unroll
                for (int q = j * PIECES / NOPS; q < (j + 1) * PIECES / NOPS; ++q) piece(q);
            }
            u32x4 w0 = {wd[0], wd[1], wd[2], wd[3]}, w1 = {wd[4], wd[5], wd[6], wd[7]};
            p_cur[0] = __builtin_bit_cast(bf16x8, w0);
            p_cur[1] = __builtin_bit_cast(bf16x8, w1);
            softmax_post(s_cur, p_cur, (part[0] + part[1]) + (part[2] + part[3]));
        };

        // Step t: S(t+1) from half ku of K stage ks into s_next, softmax of
        // s_cur into p_cur, O^T += V(t-1)^T p_prev from half vu of V stage vs.
        // FULL: all three are due, so they form one straight-line block.
        auto step = [&](int t, const unsigned char* ks, int ku, const unsigned char* vs, int vu,
                        f32x16& s_next, f32x16& s_cur, bf16x8 (&p_cur)[2], bf16x8 (&p_prev)[2],
                        auto full_tag) __attribute__((always_inline)) {
            if constexpr (decltype(full_tag)::value) {
                if (rescale_pend) apply_rescale();
                softmax_pre(s_cur, t);
                fused_step(ks, ku, vs, vu, s_next, s_cur, p_cur, p_prev);
            } else {
                const bool do_pv = t >= 1 && t - 1 < n_w;
                if (do_pv && rescale_pend) apply_rescale();
                if (t + 1 < n_w) s_mfma(ks, ku, s_next);
                if (do_pv) pv_mfma(vs, vu, p_prev);
                if (t < n_w) {
                    softmax_pre(s_cur, t);
                    const float part = exp_pack(s_cur, p_cur, m_run == kNegInf ? 0.0f : -m_run);
                    softmax_post(s_cur, p_cur, part);
                }
            }
        };

        // Stage iteration i (steps 2i + 1 and 2i + 2): reads K stage i + 1
        // and V stage i from LDS.  After the barrier (every wave's LDS stores
        // of the previous iteration are complete, and nothing reads the slots
        // of K(i) and V(i - 1) any more) it stores the registers holding
        // K(i + 2) and V(i + 1) into those slots and starts loading K(i + 3)
        // and V(i + 2): a load has a whole stage iteration to arrive.
        auto stage_iter = [&](int i, auto slot_tag) __attribute__((always_inline)) {
            constexpr int S = decltype(slot_tag)::value;
            wait_lgkmcnt0();
            barrier_no_fence();
            store_stage(kslot(Tag<S>{}), stK);
            store_stage(vslot(Tag<S + 1>{}), stV);
            load_stage(true, i + 3, stK);
            load_stage(false, i + 2, stV);
            const unsigned char* ks = kslot(Tag<S + 1>{});
            const unsigned char* vs = vslot(Tag<S>{});
            const int t1 = 2 * i + 1, t2 = 2 * i + 2;
            if (t1 + 1 < n_w) step(t1, ks, 0, vs, 0, sA, sB, pB, pA, std::true_type{});
            else step(t1, ks, 0, vs, 0, sA, sB, pB, pA, std::false_type{});
            if (t2 + 1 < n_w) step(t2, ks, 1, vs, 1, sB, sA, pA, pB, std::true_type{});
            else step(t2, ks, 1, vs, 1, sB, sA, pA, pB, std::false_type{});
        };

        // Prologue: K(0), V(0) and K(1) into LDS, K(2) and V(1) in flight,
        // then S(0) and step 0 from K stage 0.
        {
            uint4 k1[LPS];
            load_stage(true, 0, stK);
            load_stage(false, 0, stV);
            load_stage(true, 1, k1);
            flip_q();
            store_stage(k_r0, stK);
            store_stage(v_r0, stV);
            store_stage(k_r1, k1);
        }
        load_stage(true, 2, stK);
        load_stage(false, 1, stV);
        wait_lgkmcnt0();
        barrier_no_fence();
        if (n_w > 0) s_mfma(k_r0, 0, sA);
        step(0, k_r0, 1, v_r0, 0, sB, sA, pA, pB, std::false_type{});
        for (int i = 0; i < n_iters; i += RING) {
            stage_iter(i, Tag<0>{});
            if (i + 1 >= n_iters) break;
            stage_iter(i + 1, Tag<1>{});
        }
        // Every wave is done with this item's LDS before the next item's
        // prologue stores.
        barrier_no_fence();

        // ---- a7: epilogue, O = acc / l: the only device-memory write.
        const float l_tot = half_sum(l_run);
        const float inv = 1.0f / l_tot;
        if (qrow < Nq) {
            const size_t obase = (size_t)A.o_head(bh) + (size_t)qrow * A.orow();
#pragma unroll
            for (int b = 0; b < D / 32; ++b) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int dv = dv_of<D>(b, g * 8 + half * 4);
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
}

template <int D, bool CAUSAL, bool OUT_BF16, bool STRIDED>
hipError_t launch(const Problem& p, hipStream_t stream) {
    auto kernel = prefill_pipe_kernel<D, CAUSAL, OUT_BF16, STRIDED>;
    static const int per_cu = [&] {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, THREADS, 0) != hipSuccess) n = 1;
        return n > 0 ? n : 1;
    }();
    int cus = 0;
    const hipError_t e = device_cus(stream, cus);
    if (e != hipSuccess) return e;
    const int n_qtiles = (p.nq + BMQ - 1) / BMQ;
    const long long items = (long long)p.bh * n_qtiles;
    const unsigned grid = (unsigned)std::min<long long>(items, (long long)cus * per_cu);
    return launch_kernel(kernel, dim3(grid), dim3(THREADS), stream,
                         static_cast<const u16*>(p.q), static_cast<const u16*>(p.k),
                         static_cast<const u16*>(p.v), p.o, p.lse, p.nq, p.nk, p.bh, n_qtiles,
                         p.scale * kLog2e, p.lay);
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

hipError_t launch_prefill_bf16_pipe(const Problem& p, hipStream_t stream) {
    if (p.d == 64) return launch_d<64>(p, stream);
    if (p.d == 128) return launch_d<128>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace moa
