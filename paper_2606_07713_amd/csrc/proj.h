// Internal launch interface of the input-projection kernel (proj.hip).
#pragma once

#include <hip/hip_runtime_api.h>

namespace moa {

// X [m][dm] bf16 with m = B*n tokens; w[p] = the transposed weight of
// projection p (Q, K, V), [h*d][dm] bf16; out[p] = [B][h][n][d] bf16.
// dm is a multiple of 64; the caller checks sizes against 32-bit offsets.
struct ProjProblem {
    const void* x;
    const void* w[3];
    void* out[3];
    int m, n, dm, h, d;
};

hipError_t launch_proj(const ProjProblem& p, hipStream_t stream);

}  // namespace moa
