// Pieces shared by the bf16 prefill kernels: LDS tile layout (swizzle and the
// O^T row order), the persistent work schedule and the device query that
// sizes a persistent grid.
#pragma once

#include <atomic>
#include <stdint.h>

#include "device_common.h"
#include "launch.h"

namespace moa {
namespace pf {

constexpr int WAVES = 8;                     // waves per workgroup
constexpr int THREADS = WAVES * 64;
constexpr int BN = 64;                       // key rows per LDS tile
constexpr float kRescaleSlack = 8.0f;        // log2 units a tile may exceed the reference by
// A raised reference is set this far (log2 units) above the tile max that
// raised it.  Weights then start at most 2^-32, which costs no precision (bf16
// and fp32 share the exponent range; only keys ~94 units below the max would
// flush to zero, far below fp32 resolution of the sum), and later tiles must
// exceed the new reference by the fast-step limit before it is raised again:
// with wide logits the first tiles' max is typically tens of units below the
// row max, and each raise costs a redone tile.
constexpr float kRefHeadroom = 32.0f;
constexpr float kFastSumLimit = 1048576.0f;  // 2^20: partial sum bound of the fast step

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

template <int D>
struct Cfg {
    static constexpr int CHUNKS = D / 8;                        // 16-byte chunks per row
    static constexpr uint32_t ROW_BYTES = D * 2;
    static constexpr uint32_t TILE_BYTES = BN * ROW_BYTES;      // one K or V tile
};

// 16-byte-chunk XOR swizzle of LDS row `row` (a permutation of the row's
// chunks).  With 64 four-byte banks: the K operand reads (16 lanes, 16
// consecutive rows, one logical chunk) hit 16 distinct bank groups, and the
// transposing V reads (32 lanes: 4 rows x 2 chunks x 2 halves per 16 lanes)
// hit 64 distinct banks -- for d = 128 together with the dv order below.
template <int D>
__device__ __forceinline__ int swz(int row) {
    if constexpr (D == 128) return ((row & 3) << 1) | (((row >> 2) & 1) << 3) | ((row >> 3) & 1);
    return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}

// dv index held by row m (0..31) of the b-th O^T accumulator block.  For d =
// 128 the two 16-row halves of a block take dv ranges 64 apart, so the two
// 16-lane groups of a transposing read touch opposite bank halves.
template <int D>
__device__ __forceinline__ int dv_of(int b, int m) {
    if constexpr (D == 128) return (m < 16) ? 16 * b + m : 64 + 16 * b + (m - 16);
    return 32 * b + m;
}

// Persistent schedule.  The grid holds as many workgroups as the GPU runs at
// once (P); workgroup p walks its share of the n_bh * n_qtiles work items
// (head slice, query tile) and returns when it has none left, so no workgroup
// is ever dispatched behind a busy one.  Items are ranked query tile by query
// tile, all head slices of a rank together.  Without a causal mask every item
// costs the same and a workgroup takes every P-th item; with the mask, tiles
// cost in proportion to their row index, ranks run from the last query tile
// down and the deal snakes (p, 2P - 1 - p, 2P + p, ...), so every workgroup
// pairs a heavy item with a light one.
//
// Workgroups reach the 8 XCDs round-robin (p on XCD p % 8) and each XCD has
// its own L2.  When head slices and workgroups both split evenly over the
// XCDs, the deal is done per XCD over the head slices h = x (mod 8), so each
// XCD streams the K/V of only its own heads.
__device__ __forceinline__ bool item_of(int p, int i, int P, int n_bh, int n_qtiles, bool causal,
                                        int& bh, int& qt) {
    constexpr int kXcds = 8;
    int pl = p, Pl = P, hl = n_bh, x = 0, hstride = 1;
    if (n_bh % kXcds == 0 && P % kXcds == 0) {
        x = p % kXcds;
        pl = p / kXcds;
        Pl = P / kXcds;
        hl = n_bh / kXcds;
        hstride = kXcds;
    }
    const long long j = (long long)i * Pl + ((causal && (i & 1)) ? Pl - 1 - pl : pl);
    if (j >= (long long)hl * n_qtiles) return false;
    const int rank = (int)(j / hl);
    bh = x + hstride * (int)(j - (long long)rank * hl);
    qt = causal ? n_qtiles - 1 - rank : rank;
    return true;
}

// Element offsets as the kernels use them: the general strided Layout, or
// (STRIDED = false) the contiguous [B][H][N][d] layout with compile-time row
// strides, which keeps the stride arithmetic out of the registers of the
// common case.
template <int D, bool STRIDED>
struct Addr {
    const Layout& L;
    int Nq, Nk;
    __device__ __forceinline__ long long q_head(int bh) const {
        if constexpr (STRIDED) return head_offset(bh, L.H, L.qb, L.qh);
        return (long long)bh * Nq * D;
    }
    __device__ __forceinline__ long long k_head(int bh) const {
        if constexpr (STRIDED) return head_offset(bh, L.H, L.kb, L.kh);
        return (long long)bh * Nk * D;
    }
    __device__ __forceinline__ long long v_head(int bh) const {
        if constexpr (STRIDED) return head_offset(bh, L.H, L.vb, L.vh);
        return (long long)bh * Nk * D;
    }
    __device__ __forceinline__ long long o_head(int bh) const {
        if constexpr (STRIDED) return head_offset(bh, L.H, L.ob, L.oh);
        return (long long)bh * Nq * D;
    }
    __device__ __forceinline__ int qr() const { if constexpr (STRIDED) return L.qr; return D; }
    __device__ __forceinline__ int kr() const { if constexpr (STRIDED) return L.kr; return D; }
    __device__ __forceinline__ int vr() const { if constexpr (STRIDED) return L.vr; return D; }
    __device__ __forceinline__ int orow() const { if constexpr (STRIDED) return L.orow; return D; }
};

// s_waitcnt with vmcnt(N) and the other counters left alone (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt lgkmcnt(0) only: this wave's LDS accesses have completed.
__device__ __forceinline__ void wait_lgkmcnt0() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}

// Workgroup barrier without the memory-model fences of __syncthreads(): the
// release fence would also wait for every outstanding global load
// (vmcnt(0)) and so drain a prefetch pipeline at each use.  Callers order
// LDS themselves: a wave waits for its own LDS stores (or direct-to-LDS
// loads) of data others are about to read before the barrier, and every LDS
// read issued before the barrier has been consumed before it.  The signal
// fences only keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void barrier_no_fence() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Compute units of the device that runs `stream` (cached per device).
inline hipError_t device_cus(hipStream_t stream, int& cus) {
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cache[kMaxDevices];
    hipDevice_t dev = 0;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < kMaxDevices && (cus = cache[dev].load(std::memory_order_relaxed)) > 0)
        return hipSuccess;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    if (cus < 1) cus = 1;
    if (dev >= 0 && dev < kMaxDevices) cache[dev].store(cus, std::memory_order_relaxed);
    return hipSuccess;
}

}  // namespace pf
}  // namespace moa
