// C-ABI front end of the attention library: argument validation, workspace
// sizing and kernel dispatch.  Everything here is host code; it allocates no
// device memory and never synchronises.
#include <cmath>
#include <cstdint>
#include <limits>

#include "../../include/moa_attn.h"
#include "launch.h"
#include "proj.h"

namespace {

constexpr int kMaxSplits = 256;
// Keys a decode workgroup should stream at least, and the workgroup count the
// automatic split choice aims for: one per compute unit of an MI355X (256).
// Fewer, longer key chunks stream faster than many short ones, e.g. 4 splits
// of B8 H8 Nk 65536 read 7.1 TB/s against 6.0 with 128, 8 splits of B1 H32
// Nk 131072 6.6 against 5.1 with 256; grids of 256 or more rows take one
// split.  (A constant: the workspace size query has no device to ask.)
constexpr int64_t kMinKeysPerSplit = 256;
constexpr int64_t kTargetDecodeBlocks = 256;
// Prefill (Nq > 1, bf16): keys are split across workgroups when fewer than
// kPrefillSplitBelowItems 256-query items exist (half the 256 compute units
// of an MI355X), aiming at kPrefillTargetBlocks 128-query split items, each
// split covering at least kMinKeysPerPrefillSplit keys.
constexpr int64_t kPrefillSplitBelowItems = 128;
constexpr int64_t kPrefillTargetBlocks = 256;
constexpr int64_t kMinKeysPerPrefillSplit = 1024;

bool dims_ok(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv) {
    return B >= 0 && H >= 0 && Nq >= 0 && Nk >= 1 && dk >= 1 && dv >= 1;
}

bool head_supported(int64_t dk, int64_t dv) { return dk == dv && (dk == 64 || dk == 128); }

// In-head offsets are 32-bit in the kernels; grids are 1-D.
bool sizes_fit(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d) {
    const int64_t lim = std::numeric_limits<int32_t>::max();
    if (Nq > lim / d || Nk > lim / d) return false;
    if (B != 0 && H > lim / B) return false;
    const int64_t bh = B * H;
    const int64_t qtiles = (Nq + moa::kPrefillF32RowsPerBlock - 1) / moa::kPrefillF32RowsPerBlock;
    if (bh != 0 && qtiles > lim / bh) return false;
    if (bh != 0 && kMaxSplits > lim / bh) return false;
    return true;
}

int pick_splits(int64_t bh, int64_t Nk, int requested) {
    if (requested > 0) return requested;
    int64_t s = (kTargetDecodeBlocks + bh - 1) / (bh > 0 ? bh : 1);
    const int64_t cap = (Nk + kMinKeysPerSplit - 1) / kMinKeysPerSplit;
    if (s > cap) s = cap;
    if (s > kMaxSplits) s = kMaxSplits;
    if (s < 1) s = 1;
    return (int)s;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int pick_prefill_splits(int64_t bh, int64_t Nq, int64_t Nk, int requested) {
    if (requested > 0) return requested;
    if (bh * ((Nq + 255) / 256) >= kPrefillSplitBelowItems) return 1;
    const int64_t items = bh * ((Nq + 127) / 128);
    int64_t s = (kPrefillTargetBlocks + items - 1) / items;
    const int64_t cap = Nk / kMinKeysPerPrefillSplit;
    if (s > cap) s = cap;
    if (s > kMaxSplits) s = kMaxSplits;
    if (s < 1) s = 1;
    return (int)s;
}

// Split-K work items (128-query tiles x splits per head slice) must fit the
// kernels' 32-bit counters.
bool prefill_splits_fit(int64_t bh, int64_t Nq, int splits) {
    return bh * ((Nq + 127) / 128) * splits <= std::numeric_limits<int32_t>::max();
}

size_t prefill_ws_bytes(int64_t bh, int64_t Nq, int64_t d, int splits) {
    return align256((size_t)bh * (size_t)Nq * (size_t)splits * (size_t)(d + 2) * sizeof(float));
}

// Name of the HIP error behind the last MOA_ERR_HIP returned on this thread.
thread_local const char* g_last_hip_error = "hipSuccess";

// A decode call with one split writes O directly and needs no workspace.
size_t decode_ws_bytes(int64_t bh, int64_t d, int splits) {
    if (splits <= 1) return 0;
    return align256((size_t)bh * (size_t)splits * (size_t)(d + 2) * sizeof(float));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
    if (an == 0 || bn == 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bn && b0 < a0 + an;
}

// Element strides of one tensor over (batch, head, row); d is contiguous.
struct Strides {
    int64_t b, h, r;
};

Strides contiguous(int64_t H, int64_t N, int64_t d) { return {H * N * d, N * d, d}; }

// Checks of one tensor's strides: non-negative, every row 16-byte aligned,
// rows of d elements that do not overlap, and in-head byte offsets that fit
// the kernels' 32-bit descriptors.  0 = fine, else a status code.
int check_strides(const Strides& s, int64_t N, int64_t d, size_t es) {
    if (s.b < 0 || s.h < 0 || s.r < 0) return MOA_ERR_INVALID_ARG;
    if (N > 1 && s.r < d) return MOA_ERR_INVALID_ARG;
    if ((s.b * (int64_t)es) % 16 || (s.h * (int64_t)es) % 16 || (s.r * (int64_t)es) % 16)
        return MOA_ERR_UNSUPPORTED;
    const int64_t lim = std::numeric_limits<int32_t>::max();
    if (s.r > lim / (int64_t)es) return MOA_ERR_UNSUPPORTED;
    if (N > 0 && ((N - 1) * s.r + d) > lim / (int64_t)es) return MOA_ERR_UNSUPPORTED;
    return 0;
}

// Bytes from a tensor's base pointer to the end of its last element.
size_t extent_bytes(const Strides& s, int64_t B, int64_t H, int64_t N, int64_t d, size_t es) {
    if (B == 0 || H == 0 || N == 0 || d == 0) return 0;
    return (size_t)((B - 1) * s.b + (H - 1) * s.h + (N - 1) * s.r + d) * es;
}

// True if no two (batch, head, row, element) positions share an address:
// the dimensions of size > 1, by increasing stride, nest without overlap.
bool injective(const Strides& s, int64_t B, int64_t H, int64_t N, int64_t d) {
    if (B == 0 || H == 0 || N == 0) return true;   // nothing is written
    struct Dim { int64_t stride, count; } dims[3] = {{s.b, B}, {s.h, H}, {s.r, N}};
    for (int i = 0; i < 3; ++i)
        for (int j = i + 1; j < 3; ++j)
            if (dims[j].stride < dims[i].stride) { Dim t = dims[i]; dims[i] = dims[j]; dims[j] = t; }
    int64_t span = d;   // elements covered by the inner dimensions so far
    for (int i = 0; i < 3; ++i) {
        if (dims[i].count <= 1) continue;
        if (dims[i].stride < span) return false;
        span = dims[i].stride * dims[i].count;
    }
    return true;
}

// Element strides of one tensor over (batch, head, row, head element), for
// moa_attn_fwd_onf.
struct Strides4 {
    int64_t s[4];
};

Strides4 contiguous4(int64_t H, int64_t N, int64_t d) { return {{H * N * d, N * d, d, 1}}; }

// Bytes from a tensor's base pointer to the end of its last element.
size_t extent4(const Strides4& t, int64_t B, int64_t H, int64_t N, int64_t d, size_t es) {
    if (B == 0 || H == 0 || N == 0 || d == 0) return 0;
    return (size_t)((B - 1) * t.s[0] + (H - 1) * t.s[1] + (N - 1) * t.s[2] + (d - 1) * t.s[3] + 1) * es;
}

// True if no two (batch, head, row, element) positions share an address: the
// dimensions of size > 1, by increasing stride, nest without overlap.
bool injective4(const Strides4& t, int64_t B, int64_t H, int64_t N, int64_t d) {
    if (B == 0 || H == 0 || N == 0 || d == 0) return true;
    struct Dim { int64_t stride, count; } dims[4] = {{t.s[0], B}, {t.s[1], H}, {t.s[2], N}, {t.s[3], d}};
    for (int i = 0; i < 4; ++i)
        for (int j = i + 1; j < 4; ++j)
            if (dims[j].stride < dims[i].stride) { Dim x = dims[i]; dims[i] = dims[j]; dims[j] = x; }
    int64_t span = 1;   // elements covered by the inner dimensions so far
    for (int i = 0; i < 4; ++i) {
        if (dims[i].count <= 1) continue;
        if (dims[i].stride < span) return false;
        span = dims[i].stride * dims[i].count;
    }
    return true;
}

}  // namespace

extern "C" {

int moa_attn_num_splits(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                        int num_splits) {
    if (!dims_ok(B, H, Nq, Nk, dk, dv) || Nq == 0) return 1;
    if (num_splits < 0 || num_splits > kMaxSplits) return 1;
    if (Nq == 1) return pick_splits(B * H, Nk, num_splits);
    if (B * H == 0) return 1;
    return pick_prefill_splits(B * H, Nq, Nk, num_splits);
}

size_t moa_attn_workspace_bytes(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk,
                                int64_t dv, int num_splits) {
    if (!dims_ok(B, H, Nq, Nk, dk, dv) || Nq == 0) return 0;
    if (num_splits < 0 || num_splits > kMaxSplits) return 0;
    if (!head_supported(dk, dv) || !sizes_fit(B, H, Nq, Nk, dk)) return 0;
    const int64_t bh = B * H;
    if (bh == 0) return 0;
    if (Nq == 1) return decode_ws_bytes(bh, dk, pick_splits(bh, Nk, num_splits));
    const int s = pick_prefill_splits(bh, Nq, Nk, num_splits);
    if (s <= 1 || !prefill_splits_fit(bh, Nq, s)) return 0;
    return prefill_ws_bytes(bh, Nq, dk, s);
}

}  // extern "C"

namespace {

int fwd_impl(const void* Q, const void* K, const void* V, void* O, float* LSE, int64_t B, int64_t H,
             int64_t Nq, int64_t Nk, int64_t dk, int64_t dv, const int64_t* q_strides,
             const int64_t* k_strides, const int64_t* v_strides, const int64_t* o_strides,
             float scale, int causal, int in_dtype, int out_dtype, void* workspace,
             size_t workspace_bytes, int num_splits, void* stream, bool use_scratch = false) {
    // use_scratch: the library's fixed scratch array serves as the workspace
    // (moa_attn_fwd_noalloc); its device address is looked up only after the
    // validation below, and nothing is allocated.
    if (use_scratch) {
        workspace = nullptr;
        workspace_bytes = moa::kNoallocScratchBytes;
    }
    const int short_ws = use_scratch ? MOA_ERR_SCRATCH : MOA_ERR_WORKSPACE;
    auto ws_fits = [&](size_t need) {
        return use_scratch ? need <= workspace_bytes : (workspace && workspace_bytes >= need);
    };
    // ---- validation: no HIP call happens before all of it has passed
    if (!Q || !K || !V || !O) return MOA_ERR_INVALID_ARG;
    if (!dims_ok(B, H, Nq, Nk, dk, dv)) return MOA_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return MOA_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return MOA_ERR_INVALID_ARG;
    if (causal && Nq > Nk) return MOA_ERR_INVALID_ARG;
    if (in_dtype != MOA_F32 && in_dtype != MOA_BF16) return MOA_ERR_INVALID_ARG;
    if (out_dtype != MOA_F32 && out_dtype != in_dtype) return MOA_ERR_INVALID_ARG;
    if (num_splits < 0 || num_splits > kMaxSplits) return MOA_ERR_INVALID_ARG;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O) ||
        (LSE && !aligned16(LSE)) || (workspace && !aligned16(workspace)))
        return MOA_ERR_INVALID_ARG;
    if (!head_supported(dk, dv)) return MOA_ERR_UNSUPPORTED;
    if (!sizes_fit(B, H, Nq, Nk, dk)) return MOA_ERR_UNSUPPORTED;

    const size_t ies = in_dtype == MOA_F32 ? 4 : 2;
    const size_t oes = out_dtype == MOA_F32 ? 4 : 2;
    const Strides sq = q_strides ? Strides{q_strides[0], q_strides[1], q_strides[2]}
                                 : contiguous(H, Nq, dk);
    const Strides sk = k_strides ? Strides{k_strides[0], k_strides[1], k_strides[2]}
                                 : contiguous(H, Nk, dk);
    const Strides sv = v_strides ? Strides{v_strides[0], v_strides[1], v_strides[2]}
                                 : contiguous(H, Nk, dv);
    const Strides so = o_strides ? Strides{o_strides[0], o_strides[1], o_strides[2]}
                                 : contiguous(H, Nq, dv);
    int st;
    if ((st = check_strides(sq, Nq, dk, ies)) || (st = check_strides(sk, Nk, dk, ies)) ||
        (st = check_strides(sv, Nk, dv, ies)) || (st = check_strides(so, Nq, dv, oes)))
        return st;
    if (!injective(so, B, H, Nq, dv)) return MOA_ERR_INVALID_ARG;

    const int64_t bh = B * H;
    const size_t qn = extent_bytes(sq, B, H, Nq, dk, ies), kn = extent_bytes(sk, B, H, Nk, dk, ies);
    const size_t vn = extent_bytes(sv, B, H, Nk, dv, ies), on = extent_bytes(so, B, H, Nq, dv, oes);
    const size_t ln = LSE ? (size_t)bh * Nq * sizeof(float) : 0;
    if (overlaps(O, on, Q, qn) || overlaps(O, on, K, kn) || overlaps(O, on, V, vn))
        return MOA_ERR_INVALID_ARG;
    if (LSE && (overlaps(LSE, ln, O, on) || overlaps(LSE, ln, Q, qn) ||
                overlaps(LSE, ln, K, kn) || overlaps(LSE, ln, V, vn)))
        return MOA_ERR_INVALID_ARG;

    const bool decode = (Nq == 1);
    int splits = 1;
    size_t need = 0;
    if (decode && bh > 0) {
        splits = pick_splits(bh, Nk, num_splits);
        need = decode_ws_bytes(bh, dk, splits);
        if (need && !ws_fits(need)) return short_ws;
    } else if (!decode && bh > 0 && Nq > 0 && in_dtype == MOA_BF16) {
        // Split-K prefill: explicitly requested splits need the workspace;
        // the automatic choice falls back to one pass without it.
        splits = pick_prefill_splits(bh, Nq, Nk, num_splits);
        if (splits > 1 && !prefill_splits_fit(bh, Nq, splits)) return MOA_ERR_UNSUPPORTED;
        need = splits > 1 ? prefill_ws_bytes(bh, Nq, dk, splits) : 0;
        if (need && !ws_fits(need)) {
            if (num_splits > 1) return short_ws;
            splits = 1;
            need = 0;
        }
    }
    if (need && !use_scratch) {
        const size_t wn = need;
        if (overlaps(workspace, wn, O, on) || overlaps(workspace, wn, Q, qn) ||
            overlaps(workspace, wn, K, kn) || overlaps(workspace, wn, V, vn) ||
            (LSE && overlaps(workspace, wn, LSE, ln)))
            return MOA_ERR_INVALID_ARG;
    }
    if (bh == 0 || Nq == 0) return MOA_OK;
    if (use_scratch && need) {
        const hipError_t e = moa::noalloc_scratch(static_cast<hipStream_t>(stream), &workspace);
        if (e != hipSuccess) {
            g_last_hip_error = hipGetErrorName(e);
            return MOA_ERR_HIP;
        }
    }

    moa::Problem p;
    p.q = Q; p.k = K; p.v = V; p.o = O; p.lse = LSE;
    p.bh = (int)bh; p.nq = (int)Nq; p.nk = (int)Nk; p.d = (int)dk;
    p.scale = scale;
    p.causal = causal != 0;
    p.in_bf16 = in_dtype == MOA_BF16;
    p.out_bf16 = out_dtype == MOA_BF16;
    p.lay.qb = sq.b; p.lay.qh = sq.h; p.lay.qr = (int)sq.r;
    p.lay.kb = sk.b; p.lay.kh = sk.h; p.lay.kr = (int)sk.r;
    p.lay.vb = sv.b; p.lay.vh = sv.h; p.lay.vr = (int)sv.r;
    p.lay.ob = so.b; p.lay.oh = so.h; p.lay.orow = (int)so.r;
    p.lay.H = (int)H;
    p.splits = splits;
    p.ws = static_cast<float*>(workspace);
    hipStream_t s = static_cast<hipStream_t>(stream);

    hipError_t e;
    if (decode)
        e = moa::launch_decode(p, splits, static_cast<float*>(workspace), s);
    else if (p.in_bf16)
        e = moa::launch_prefill_bf16(p, s);
    else
        e = moa::launch_prefill_f32(p, s);
    if (e != hipSuccess) {
        g_last_hip_error = hipGetErrorName(e);
        return MOA_ERR_HIP;
    }
    return MOA_OK;
}

}  // namespace

extern "C" {

int moa_attn_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE, int64_t B,
                 int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv, float scale,
                 int causal, int in_dtype, int out_dtype, void* workspace,
                 size_t workspace_bytes, int num_splits, void* stream) {
    return fwd_impl(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, nullptr, nullptr, nullptr, nullptr,
                    scale, causal, in_dtype, out_dtype, workspace, workspace_bytes, num_splits,
                    stream);
}

int moa_attn_fwd_strided(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                         const int64_t* q_strides, const int64_t* k_strides,
                         const int64_t* v_strides, const int64_t* o_strides, float scale,
                         int causal, int in_dtype, int out_dtype, void* workspace,
                         size_t workspace_bytes, int num_splits, void* stream) {
    return fwd_impl(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, q_strides, k_strides, v_strides,
                    o_strides, scale, causal, in_dtype, out_dtype, workspace, workspace_bytes,
                    num_splits, stream);
}

int moa_attn_fwd_noalloc(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                         float scale, int causal, int in_dtype, int out_dtype, int num_splits,
                         void* stream) {
    return fwd_impl(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, nullptr, nullptr, nullptr, nullptr,
                    scale, causal, in_dtype, out_dtype, nullptr, 0, num_splits, stream, true);
}

int moa_attn_fwd_onf(const void* Q, const void* K, const void* V, void* O, float* LSE,
                     int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                     const int64_t* q_strides, const int64_t* k_strides, const int64_t* v_strides,
                     const int64_t* o_strides, float scale, int causal, int in_dtype,
                     int out_dtype, void* workspace, size_t workspace_bytes, int num_splits,
                     void* stream) {
    // ---- validation: no HIP call happens before all of it has passed
    if (!Q || !K || !V || !O) return MOA_ERR_INVALID_ARG;
    if (!dims_ok(B, H, Nq, Nk, dk, dv)) return MOA_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return MOA_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return MOA_ERR_INVALID_ARG;
    if (causal && Nq > Nk) return MOA_ERR_INVALID_ARG;
    if (in_dtype != MOA_F32 && in_dtype != MOA_BF16) return MOA_ERR_INVALID_ARG;
    if (out_dtype != MOA_F32 && out_dtype != in_dtype) return MOA_ERR_INVALID_ARG;
    if (num_splits < 0 || num_splits > kMaxSplits) return MOA_ERR_INVALID_ARG;
    if (!head_supported(dk, dv)) return MOA_ERR_UNSUPPORTED;
    if (!sizes_fit(B, H, Nq, Nk, dk)) return MOA_ERR_UNSUPPORTED;
    const Strides4 sq = q_strides ? Strides4{{q_strides[0], q_strides[1], q_strides[2], q_strides[3]}}
                                  : contiguous4(H, Nq, dk);
    const Strides4 sk = k_strides ? Strides4{{k_strides[0], k_strides[1], k_strides[2], k_strides[3]}}
                                  : contiguous4(H, Nk, dk);
    const Strides4 sv = v_strides ? Strides4{{v_strides[0], v_strides[1], v_strides[2], v_strides[3]}}
                                  : contiguous4(H, Nk, dv);
    const Strides4 so = o_strides ? Strides4{{o_strides[0], o_strides[1], o_strides[2], o_strides[3]}}
                                  : contiguous4(H, Nq, dv);
    for (const Strides4* t : {&sq, &sk, &sv, &so})
        for (int i = 0; i < 4; ++i)
            if (t->s[i] < 0) return MOA_ERR_INVALID_ARG;

    // Layouts the matrix-core kernels read (contiguous head elements, 16-byte
    // aligned rows, rows of d elements that do not overlap, 32-bit in-head
    // offsets) go through moa_attn_fwd_strided's path unchanged.
    const size_t ies = in_dtype == MOA_F32 ? 4 : 2;
    const size_t oes = out_dtype == MOA_F32 ? 4 : 2;
    auto fast_ok = [&](const Strides4& t, int64_t N, int64_t d, size_t es) {
        return t.s[3] == 1 && check_strides(Strides{t.s[0], t.s[1], t.s[2]}, N, d, es) == 0;
    };
    if (fast_ok(sq, Nq, dk, ies) && fast_ok(sk, Nk, dk, ies) && fast_ok(sv, Nk, dv, ies) &&
        fast_ok(so, Nq, dv, oes) && aligned16(Q) && aligned16(K) && aligned16(V) && aligned16(O)) {
        const int64_t q3[3] = {sq.s[0], sq.s[1], sq.s[2]}, k3[3] = {sk.s[0], sk.s[1], sk.s[2]};
        const int64_t v3[3] = {sv.s[0], sv.s[1], sv.s[2]}, o3[3] = {so.s[0], so.s[1], so.s[2]};
        return fwd_impl(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, q3, k3, v3, o3, scale, causal,
                        in_dtype, out_dtype, workspace, workspace_bytes, num_splits, stream);
    }

    // Element-gather path: any strides; O must not write an element twice.
    auto aligned_to = [](const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; };
    if (!aligned_to(Q, ies) || !aligned_to(K, ies) || !aligned_to(V, ies) || !aligned_to(O, oes) ||
        (LSE && !aligned_to(LSE, 4)))
        return MOA_ERR_INVALID_ARG;
    if (!injective4(so, B, H, Nq, dv)) return MOA_ERR_INVALID_ARG;
    const int64_t bh = B * H;
    const size_t qn = extent4(sq, B, H, Nq, dk, ies), kn = extent4(sk, B, H, Nk, dk, ies);
    const size_t vn = extent4(sv, B, H, Nk, dv, ies), on = extent4(so, B, H, Nq, dv, oes);
    const size_t ln = LSE ? (size_t)bh * Nq * sizeof(float) : 0;
    if (overlaps(O, on, Q, qn) || overlaps(O, on, K, kn) || overlaps(O, on, V, vn))
        return MOA_ERR_INVALID_ARG;
    if (LSE && (overlaps(LSE, ln, O, on) || overlaps(LSE, ln, Q, qn) ||
                overlaps(LSE, ln, K, kn) || overlaps(LSE, ln, V, vn)))
        return MOA_ERR_INVALID_ARG;
    if (bh == 0 || Nq == 0) return MOA_OK;

    moa::Problem p{};
    p.q = Q; p.k = K; p.v = V; p.o = O; p.lse = LSE;
    p.bh = (int)bh; p.nq = (int)Nq; p.nk = (int)Nk; p.d = (int)dk;
    p.scale = scale;
    p.causal = causal != 0;
    p.in_bf16 = in_dtype == MOA_BF16;
    p.out_bf16 = out_dtype == MOA_BF16;
    p.splits = 1;
    moa::GatherLayout g;
    for (int i = 0; i < 4; ++i) {
        g.q[i] = sq.s[i]; g.k[i] = sk.s[i]; g.v[i] = sv.s[i]; g.o[i] = so.s[i];
    }
    g.H = (int)H;
    const hipError_t e = moa::launch_prefill_gather(p, g, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        g_last_hip_error = hipGetErrorName(e);
        return MOA_ERR_HIP;
    }
    return MOA_OK;
}

size_t moa_attn_bwd_workspace_bytes(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk,
                                    int64_t dv) {
    if (!dims_ok(B, H, Nq, Nk, dk, dv)) return 0;
    if (!head_supported(dk, dv) || !sizes_fit(B, H, Nq, Nk, dk)) return 0;
    return align256((size_t)(B * H) * (size_t)Nq * sizeof(float));
}

int moa_attn_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, void* dQ, void* dK, void* dV, int64_t B, int64_t H, int64_t Nq,
                 int64_t Nk, int64_t dk, int64_t dv, float scale, int causal, int in_dtype,
                 int o_dtype, int grad_dtype, void* workspace, size_t workspace_bytes,
                 void* stream) {
    // ---- validation: no HIP call happens before all of it has passed
    if (!dims_ok(B, H, Nq, Nk, dk, dv)) return MOA_ERR_INVALID_ARG;
    // A pointer may be NULL only when its tensor has no elements.
    const bool has_q = B * H * Nq > 0, has_k = B * H > 0;
    if ((has_k && (!K || !V || !dK || !dV)) || (has_q && (!Q || !O || !dO || !LSE || !dQ)))
        return MOA_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return MOA_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return MOA_ERR_INVALID_ARG;
    if (causal && Nq > Nk) return MOA_ERR_INVALID_ARG;
    for (int t : {in_dtype, o_dtype, grad_dtype})
        if (t != MOA_F32 && t != MOA_BF16) return MOA_ERR_INVALID_ARG;
    const void* ptrs[] = {Q, K, V, O, dO, LSE, dQ, dK, dV};
    for (const void* q : ptrs)
        if (!aligned16(q)) return MOA_ERR_INVALID_ARG;
    if (workspace && !aligned16(workspace)) return MOA_ERR_INVALID_ARG;
    if (in_dtype != MOA_BF16) return MOA_ERR_UNSUPPORTED;
    if (!head_supported(dk, dv)) return MOA_ERR_UNSUPPORTED;
    if (!sizes_fit(B, H, Nq, Nk, dk)) return MOA_ERR_UNSUPPORTED;

    const int64_t bh = B * H;
    const size_t qn = (size_t)(bh * Nq * dk) * 2, kn = (size_t)(bh * Nk * dk) * 2;
    const size_t vn = (size_t)(bh * Nk * dv) * 2, on = (size_t)(bh * Nq * dv) * (o_dtype == MOA_F32 ? 4 : 2);
    const size_t gn = (size_t)(bh * Nq * dv) * 2, ln = (size_t)(bh * Nq) * sizeof(float);
    const size_t ges = grad_dtype == MOA_F32 ? 4 : 2;
    const size_t dqn = (size_t)(bh * Nq * dk) * ges, dkn = (size_t)(bh * Nk * dk) * ges;
    const size_t dvn = (size_t)(bh * Nk * dv) * ges;
    const size_t need = moa_attn_bwd_workspace_bytes(B, H, Nq, Nk, dk, dv);
    if (need && (!workspace || workspace_bytes < need)) return MOA_ERR_WORKSPACE;
    struct Buf { const void* p; size_t n; };
    const Buf ins[] = {{Q, qn}, {K, kn}, {V, vn}, {O, on}, {dO, gn}, {LSE, ln}};
    const Buf outs[] = {{dQ, dqn}, {dK, dkn}, {dV, dvn}, {workspace, need}};
    for (int i = 0; i < 4; ++i) {
        for (const Buf& b : ins)
            if (overlaps(outs[i].p, outs[i].n, b.p, b.n)) return MOA_ERR_INVALID_ARG;
        for (int j = i + 1; j < 4; ++j)
            if (overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return MOA_ERR_INVALID_ARG;
    }
    if (bh == 0) return MOA_OK;

    moa::BwdProblem p;
    p.q = Q; p.k = K; p.v = V; p.o = O; p.dout = dO; p.lse = LSE;
    p.dsum = static_cast<float*>(workspace);
    p.dq = dQ; p.dk = dK; p.dv = dV;
    p.bh = (int)bh; p.nq = (int)Nq; p.nk = (int)Nk; p.d = (int)dk;
    p.scale = scale;
    p.causal = causal != 0;
    p.o_bf16 = o_dtype == MOA_BF16;
    p.grad_bf16 = grad_dtype == MOA_BF16;
    const hipError_t e = moa::launch_bwd(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        g_last_hip_error = hipGetErrorName(e);
        return MOA_ERR_HIP;
    }
    return MOA_OK;
}

size_t moa_attn_proj_workspace_bytes(int64_t B, int64_t N, int64_t Dm, int64_t H, int64_t d) {
    if (B < 0 || N < 0 || Dm < 1 || H < 0 || !head_supported(d, d) || Dm % 64) return 0;
    if (!sizes_fit(B, H, N, N, d)) return 0;
    const size_t qkv = align256((size_t)(B * H * N * d) * 2);
    const size_t att = N > 0 ? moa_attn_workspace_bytes(B, H, N, N, d, d, 0) : 0;
    return 3 * qkv + att;
}

int moa_attn_fwd_proj(const void* X, const void* Wq, const void* Wk, const void* Wv, void* O,
                      float* LSE, int64_t B, int64_t N, int64_t Dm, int64_t H, int64_t d,
                      float scale, int causal, int out_dtype, void* workspace,
                      size_t workspace_bytes, void* stream) {
    // ---- validation: no HIP call happens before all of it has passed
    if (B < 0 || N < 0 || H < 0 || Dm < 1 || d < 1) return MOA_ERR_INVALID_ARG;
    const int64_t bh = B * H, tokens = B * N;
    const bool any = bh > 0 && N > 0;
    if (any && (!X || !Wq || !Wk || !Wv || !O)) return MOA_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return MOA_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return MOA_ERR_INVALID_ARG;
    if (out_dtype != MOA_F32 && out_dtype != MOA_BF16) return MOA_ERR_INVALID_ARG;
    const void* ptrs[] = {X, Wq, Wk, Wv, O, LSE, workspace};
    for (const void* q : ptrs)
        if (!aligned16(q)) return MOA_ERR_INVALID_ARG;
    if (!head_supported(d, d)) return MOA_ERR_UNSUPPORTED;
    if (Dm % 64) return MOA_ERR_UNSUPPORTED;
    if (!sizes_fit(B, H, N, N, d)) return MOA_ERR_UNSUPPORTED;
    const int64_t lim = std::numeric_limits<int32_t>::max();
    if (tokens > lim || H * d > lim / 3 || (tokens > 0 && Dm > lim / tokens)) return MOA_ERR_UNSUPPORTED;
    if (!any) return MOA_OK;

    const size_t need = moa_attn_proj_workspace_bytes(B, N, Dm, H, d);
    if (!workspace || workspace_bytes < need) return MOA_ERR_WORKSPACE;
    const size_t xn = (size_t)(tokens * Dm) * 2, wn = (size_t)(H * d * Dm) * 2;
    const size_t on = (size_t)(bh * N * d) * (out_dtype == MOA_F32 ? 4 : 2);
    const size_t ln = LSE ? (size_t)(bh * N) * sizeof(float) : 0;
    struct Buf { const void* p; size_t n; };
    const Buf ins[] = {{X, xn}, {Wq, wn}, {Wk, wn}, {Wv, wn}};
    const Buf outs[] = {{O, on}, {LSE, ln}, {workspace, need}};
    for (int i = 0; i < 3; ++i) {
        for (const Buf& b : ins)
            if (overlaps(outs[i].p, outs[i].n, b.p, b.n)) return MOA_ERR_INVALID_ARG;
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return MOA_ERR_INVALID_ARG;
    }

    // Q, K, V (bf16, [B][H][N][d]) and the attention's own workspace.
    const size_t qkv = align256((size_t)(bh * N * d) * 2);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    moa::ProjProblem pp;
    pp.x = X;
    pp.w[0] = Wq; pp.w[1] = Wk; pp.w[2] = Wv;
    for (int i = 0; i < 3; ++i) pp.out[i] = ws + i * qkv;
    pp.m = (int)tokens; pp.n = (int)N; pp.dm = (int)Dm; pp.h = (int)H; pp.d = (int)d;
    const hipError_t e = moa::launch_proj(pp, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        g_last_hip_error = hipGetErrorName(e);
        return MOA_ERR_HIP;
    }
    return fwd_impl(pp.out[0], pp.out[1], pp.out[2], O, LSE, B, H, N, N, d, d, nullptr, nullptr,
                    nullptr, nullptr, scale, causal, MOA_BF16, out_dtype, ws + 3 * qkv,
                    need - 3 * qkv, 0, stream);
}

const char* moa_attn_last_hip_error(void) { return g_last_hip_error; }

const char* moa_attn_status_string(int status) {
    switch (status) {
        case MOA_OK: return "ok";
        case MOA_ERR_INVALID_ARG: return "invalid argument";
        case MOA_ERR_UNSUPPORTED: return "unsupported head size or problem size";
        case MOA_ERR_WORKSPACE: return "workspace missing or too small";
        case MOA_ERR_HIP: return "HIP runtime error while enqueueing";
        case MOA_ERR_SCRATCH:
            return "problem needs more scratch than the library's fixed array holds "
                   "(MOA_NOALLOC_SCRATCH_BYTES); use moa_attn_fwd with a workspace";
        default: return "unknown status";
    }
}

}  // extern "C"
