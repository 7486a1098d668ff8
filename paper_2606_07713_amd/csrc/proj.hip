// Input projections Q = X W_Q, K = X W_K, V = X W_V (the paper's problem
// statement) on gfx950 matrix cores, written straight into the head-split
// [B][H][N][d] layout the attention kernels read.
//
// One launch computes all three projections as one matrix product
//   C^T[f][m] = sum_k Wt[f][k] * X[m][k],   m = b*N + n,  f = p*H*d + h*d + e,
// where Wt = [Wq; Wk; Wv] holds the weights transposed ([H*d][Dm] each, the
// layout of a dense layer's weight) and p selects the projection.  Both
// operands are read along k, their stored order, so neither is transposed.
// C^T orientation: the MFMA A operand is a weight row, the B operand an X
// row, and each lane's accumulator holds 4-feature runs of one token, which
// are stored as 8-byte bf16 groups (round to nearest even).
//
// Tiling: a workgroup of 8 waves owns a 256-feature x 256-token tile and walks
// k in steps of 64.  Each step's two tiles (32 KB each) are loaded from device
// memory into registers one step ahead and stored into a two-stage LDS ring
// (16-byte chunks XOR-swizzled per row, conflict-free for both the stores and
// the operand reads); each wave multiplies a 128 x 64 sub-tile (4 x 2 blocks
// of v_mfma_f32_32x32x16_bf16, fp32 accumulation).  A 256 x 256 tile does
// 128 flops per byte it loads, which keeps the load rate of a fully busy
// GPU (~16 TB/s at the matrix-core peak) within what its caches deliver; a
// 128 x 128 tile needs twice that and measured at ~13% of peak.
#include "device_common.h"
#include "launch.h"
#include "proj.h"

namespace moa {
namespace {

constexpr int PT = 256;        // tile edge (features and tokens)
constexpr int PK = 64;         // k per step
constexpr int PWAVES = 8;
constexpr int PTHREADS = PWAVES * 64;
constexpr int ROWB = PK * 2;   // bytes of one tile row per step
constexpr int TILEB = PT * ROWB;
constexpr int LOADS = TILEB / (PTHREADS * 16);   // 16-byte loads per thread per tile
static_assert(LOADS == 4, "tile split");
constexpr int FB = 4, MB = 2;  // 32-row blocks per wave: features, tokens

// Physical 16-byte chunk of logical chunk c in row r (8 chunks per row):
// rows r and r ^ 1 sit in opposite bank halves, and within a half the 8
// rows that a 16-lane read group touches see 8 distinct chunks.
__device__ __forceinline__ int pswz(int r) { return (r >> 1) & 7; }

struct ProjArgs {
    const u16* x;
    const u16* w[3];
    u16* out[3];
    int M, N, Dm, H, d, F;
};

__global__ __launch_bounds__(PTHREADS, 1) void proj_kernel(ProjArgs a) {
    __shared__ __attribute__((aligned(1024))) unsigned char w_s0[TILEB];
    __shared__ __attribute__((aligned(1024))) unsigned char w_s1[TILEB];
    __shared__ __attribute__((aligned(1024))) unsigned char x_s0[TILEB];
    __shared__ __attribute__((aligned(1024))) unsigned char x_s1[TILEB];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 31, half = lane >> 5;
    const int tiles_m = (a.M + PT - 1) / PT;
    const int tm = blockIdx.x % tiles_m, tf = blockIdx.x / tiles_m;
    const int m0 = tm * PT, f0 = tf * PT;
    const int FT = 3 * a.F;

    // Per-thread load slots: chunk s = i*256 + tid of a tile -> row s / 8,
    // logical chunk s % 8; the source row is clamped into range (rows past
    // the end are loaded but never stored).
    const u16* wsrc[LOADS];
    const u16* xsrc[LOADS];
    uint32_t sw[LOADS];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int s = i * PTHREADS + tid, r = s >> 3, c = s & 7;
        const int f = min(f0 + r, FT - 1), p = f / a.F;
        const u16* wp = p == 0 ? a.w[0] : (p == 1 ? a.w[1] : a.w[2]);   // no dynamic indexing
        wsrc[i] = wp + (size_t)(f - p * a.F) * a.Dm + c * 8;
        xsrc[i] = a.x + (size_t)min(m0 + r, a.M - 1) * a.Dm + c * 8;
        sw[i] = (uint32_t)r * ROWB + (uint32_t)((c ^ pswz(r)) * 16);
    }
    u32x4 wr[LOADS], xr[LOADS];
    auto load = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            wr[i] = *reinterpret_cast<const u32x4*>(wsrc[i] + k0);
            xr[i] = *reinterpret_cast<const u32x4*>(xsrc[i] + k0);
        }
    };
    auto store = [&](unsigned char* ws, unsigned char* xs) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            *reinterpret_cast<u32x4*>(ws + sw[i]) = wr[i];
            *reinterpret_cast<u32x4*>(xs + sw[i]) = xr[i];
        }
    };

    // Operand read addresses: this wave's 128 features (A) and 64 tokens (B);
    // the k chunk 2 kk + half is added per step (the swizzle is per row, so
    // the chunk offsets are kept per block).
    const int wf = (wave >> 2) * (FB * 32), wm = (wave & 3) * (MB * 32);
    uint32_t ra[FB], rb[MB];
    int sa[FB], sb[MB];
#pragma unroll
    for (int i = 0; i < FB; ++i) {
        const int r = wf + i * 32 + col;
        ra[i] = (uint32_t)r * ROWB;
        sa[i] = pswz(r);
    }
#pragma unroll
    for (int j = 0; j < MB; ++j) {
        const int r = wm + j * 32 + col;
        rb[j] = (uint32_t)r * ROWB;
        sb[j] = pswz(r);
    }

    f32x16 acc[FB][MB];
#pragma unroll
    for (int i = 0; i < FB; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j) acc[i][j] = f32x16{};

    auto compute = [&](const unsigned char* ws, const unsigned char* xs) __attribute__((always_inline)) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const int c = 2 * kk + half;
            bf16x8 fa[FB], fb[MB];
#pragma unroll
            for (int i = 0; i < FB; ++i)
                fa[i] = *reinterpret_cast<const bf16x8*>(ws + ra[i] + ((c ^ sa[i]) << 4));
#pragma unroll
            for (int j = 0; j < MB; ++j)
                fb[j] = *reinterpret_cast<const bf16x8*>(xs + rb[j] + ((c ^ sb[j]) << 4));
#pragma unroll
            for (int i = 0; i < FB; ++i)
#pragma unroll
                for (int j = 0; j < MB; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
    };

    const int steps = a.Dm / PK;
    load(0);
    store(w_s0, x_s0);
    __syncthreads();
    for (int t = 0; t < steps; t += 2) {
        if (t + 1 < steps) load((t + 1) * PK);
        compute(w_s0, x_s0);
        if (t + 1 >= steps) break;
        store(w_s1, x_s1);
        __syncthreads();
        if (t + 2 < steps) load((t + 2) * PK);
        compute(w_s1, x_s1);
        if (t + 2 >= steps) break;
        store(w_s0, x_s0);
        __syncthreads();
    }

    // Epilogue: block (i, j) holds features wf + 32 i + 8 g + 4 half + {0..3}
    // of token wm + 32 j + col, for g = 0..3.
#pragma unroll
    for (int j = 0; j < MB; ++j) {
        const int m = m0 + wm + j * 32 + col;
        if (m >= a.M) continue;
        const int b = m / a.N, n = m - b * a.N;
#pragma unroll
        for (int i = 0; i < FB; ++i) {
            const int fb0 = f0 + wf + i * 32;        // 32 features: one projection, one head
            if (fb0 >= FT) continue;
            const int p = fb0 / a.F, fh = fb0 - p * a.F, h = fh / a.d, e0 = fh - h * a.d;
            u16* op = p == 0 ? a.out[0] : (p == 1 ? a.out[1] : a.out[2]);
            u16* dst = op + ((size_t)(b * a.H + h) * a.N + n) * a.d + e0 + 4 * half;
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<uint2*>(dst + 8 * g) =
                    make_uint2(pack_bf16x2(acc[i][j][4 * g + 0], acc[i][j][4 * g + 1]),
                               pack_bf16x2(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]));
        }
    }
}

}  // namespace

hipError_t launch_proj(const ProjProblem& p, hipStream_t stream) {
    if (p.m == 0) return hipSuccess;
    ProjArgs a;
    a.x = static_cast<const u16*>(p.x);
    for (int i = 0; i < 3; ++i) {
        a.w[i] = static_cast<const u16*>(p.w[i]);
        a.out[i] = static_cast<u16*>(p.out[i]);
    }
    a.M = p.m; a.N = p.n; a.Dm = p.dm; a.H = p.h; a.d = p.d; a.F = p.h * p.d;
    const long long tiles = (long long)((p.m + PT - 1) / PT) * ((3 * a.F + PT - 1) / PT);
    return launch_kernel(proj_kernel, dim3((unsigned)tiles), dim3(PTHREADS), stream, a);
}

}  // namespace moa
