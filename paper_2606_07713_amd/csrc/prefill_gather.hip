// Fused attention on tensors stored with arbitrary per-dimension strides,
// including a strided head dimension: column-major heads ([d][N] per head),
// rows that are not 16-byte aligned, and any mix of such layouts across Q, K,
// V and O.  These are the storage functions of the footnote to eq. gamma, with
// every access at base + sum_k stride_k * i_k (Def. "Operational Normal
// Form").
//
// The fast kernels read whole 16-byte row chunks; this one gathers element by
// element instead.  One workgroup owns 64 queries of one (batch*head); a quad
// of lanes per query splits d.  K/V tiles of 32 keys are gathered into LDS as
// fp32 (rows in order, so nothing is transposed in device memory), with the
// lanes walking the tensor's contiguous dimension: key rows for column-major
// storage, head elements otherwise.  Scores, the running max and sum and the
// weights stay in registers (eqs. dnf_attn and output_dnf); only O (and the
// optional LSE) are written.  Inputs are fp32 or bf16, all arithmetic is fp32
// with the exact online softmax per tile, so the result is within fp32
// rounding of the attention of the stored values.  Nq = 1 (decode-shaped
// calls) runs here too.  Throughput is far below the matrix-core kernels: this
// path exists for layouts they cannot read.
#include "device_common.h"
#include "launch.h"

namespace moa {
namespace {

constexpr int ROWS = 64;          // queries per workgroup
constexpr int THREADS = ROWS * 4;
constexpr int KT = 32;            // keys per tile

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, long long idx) {
    if constexpr (sizeof(T) == 4) {
        return p[idx];
    } else {
        return __uint_as_float((uint32_t)p[idx] << 16);
    }
}

// Element offset of (bh, row, e) of a tensor with strides s = {batch, head,
// row, element}.
__device__ __forceinline__ long long goff(const long long* s, int H, int bh, long long row, int e) {
    const int b = bh / H, h = bh - b * H;
    return (long long)b * s[0] + (long long)h * s[1] + row * s[2] + (long long)e * s[3];
}

template <typename T, int D, bool CAUSAL, bool OUT_BF16>
__global__ __launch_bounds__(THREADS) void prefill_gather_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    void* __restrict__ Out, float* __restrict__ LSE, int Nq, int Nk, int n_qtiles, float c,
    GatherLayout L) {
    constexpr int CH = D / 16;    // groups of 4 elements per lane: e = (j*4 + quad)*4 + {0..3}
    __shared__ __attribute__((aligned(16))) float Ks[KT * D];
    __shared__ __attribute__((aligned(16))) float Vs[KT * D];

    const int tid = threadIdx.x;
    const int quad = tid & 3;
    const int bh = blockIdx.x / n_qtiles;
    const int qt = blockIdx.x % n_qtiles;
    const int qrow = qt * ROWS + (tid >> 2);
    const int qrow_c = qrow < Nq ? qrow : Nq - 1;
    const int off = Nk - Nq;

    float4 qv[CH], acc[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        const int e0 = (j * 4 + quad) * 4;
        qv[j] = make_float4(load_elem(Q, goff(L.q, L.H, bh, qrow_c, e0)),
                            load_elem(Q, goff(L.q, L.H, bh, qrow_c, e0 + 1)),
                            load_elem(Q, goff(L.q, L.H, bh, qrow_c, e0 + 2)),
                            load_elem(Q, goff(L.q, L.H, bh, qrow_c, e0 + 3)));
        acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float m_run = kNegInf, l_run = 0.0f;

    int kv_end = Nk;
    if (CAUSAL) kv_end = min(Nk, qt * ROWS + ROWS + off);
    const int n_kt = (kv_end + KT - 1) / KT;
    // Lanes walk key rows when a tensor's head elements are strided (its rows
    // are then the contiguous dimension), head elements otherwise.
    const bool k_rows_fast = L.k[3] != 1, v_rows_fast = L.v[3] != 1;

    for (int kt = 0; kt < n_kt; ++kt) {
        const int kbase = kt * KT;
        __syncthreads();
        for (int idx = tid; idx < KT * D; idx += THREADS) {
            int row = k_rows_fast ? idx % KT : idx / D;
            int e = k_rows_fast ? idx / KT : idx % D;
            Ks[row * D + e] = load_elem(K, goff(L.k, L.H, bh, min(kbase + row, Nk - 1), e));
            row = v_rows_fast ? idx % KT : idx / D;
            e = v_rows_fast ? idx / KT : idx % D;
            Vs[row * D + e] = load_elem(V, goff(L.v, L.H, bh, min(kbase + row, Nk - 1), e));
        }
        __syncthreads();

        // scores of this tile, in log2 units (t = c * <q, k>)
        float t[KT];
        float tmax = kNegInf;
#pragma unroll
        for (int j = 0; j < KT; ++j) {
            float part = 0.0f;
#pragma unroll
            for (int h = 0; h < CH; ++h) {
                const float4 kk = *reinterpret_cast<const float4*>(&Ks[j * D + (h * 4 + quad) * 4]);
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
                const float4 vv = *reinterpret_cast<const float4*>(&Vs[j * D + (h * 4 + quad) * 4]);
                acc[h].x = __builtin_fmaf(p, vv.x, acc[h].x);
                acc[h].y = __builtin_fmaf(p, vv.y, acc[h].y);
                acc[h].z = __builtin_fmaf(p, vv.z, acc[h].z);
                acc[h].w = __builtin_fmaf(p, vv.w, acc[h].w);
            }
        }
    }

    if (qrow < Nq) {
        const float inv = 1.0f / l_run;
#pragma unroll
        for (int h = 0; h < CH; ++h) {
            const int e0 = (h * 4 + quad) * 4;
            const float o[4] = {acc[h].x * inv, acc[h].y * inv, acc[h].z * inv, acc[h].w * inv};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const long long at = goff(L.o, L.H, bh, qrow, e0 + i);
                if constexpr (OUT_BF16)
                    static_cast<u16*>(Out)[at] = (u16)f32_to_bf16_bits(o[i]);
                else
                    static_cast<float*>(Out)[at] = o[i];
            }
        }
        if (LSE != nullptr && quad == 0)
            LSE[(size_t)bh * Nq + qrow] = (m_run + __log2f(l_run)) * kLn2;
    }
}

template <typename T, int D, bool CAUSAL, bool OUT_BF16>
hipError_t launch(const Problem& p, const GatherLayout& g, hipStream_t stream) {
    const int n_qtiles = (p.nq + ROWS - 1) / ROWS;
    const long long blocks = (long long)p.bh * n_qtiles;
    return launch_kernel(prefill_gather_kernel<T, D, CAUSAL, OUT_BF16>, dim3((unsigned)blocks),
                         dim3(THREADS), stream, static_cast<const T*>(p.q),
                         static_cast<const T*>(p.k), static_cast<const T*>(p.v), p.o, p.lse, p.nq,
                         p.nk, n_qtiles, p.scale * kLog2e, g);
}

template <typename T, int D>
hipError_t launch_c(const Problem& p, const GatherLayout& g, hipStream_t stream) {
    if (p.causal)
        return p.out_bf16 ? launch<T, D, true, true>(p, g, stream) : launch<T, D, true, false>(p, g, stream);
    return p.out_bf16 ? launch<T, D, false, true>(p, g, stream) : launch<T, D, false, false>(p, g, stream);
}

template <typename T>
hipError_t launch_t(const Problem& p, const GatherLayout& g, hipStream_t stream) {
    if (p.d == 64) return launch_c<T, 64>(p, g, stream);
    if (p.d == 128) return launch_c<T, 128>(p, g, stream);
    return hipErrorInvalidValue;
}

}  // namespace

static_assert(ROWS == kPrefillGatherRowsPerBlock, "row tile mismatch");

hipError_t launch_prefill_gather(const Problem& p, const GatherLayout& g, hipStream_t stream) {
    return p.in_bf16 ? launch_t<u16>(p, g, stream) : launch_t<float>(p, g, stream);
}

}  // namespace moa
