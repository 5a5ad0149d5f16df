// tgl_cells.hpp -- the cells of a run's time directory (tgl_cell), shared
// by the T-CSR build, which writes the directory, and the sampler, which
// reads it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tgl {

// A run with first and last timestamps f <= l and K >= 1 cells splits [f, l]
// evenly.  The build and the sampler both place timestamps with these two
// functions, so a threshold and the entries it is compared with always fall
// in cells by the same float operations (each rounded to nearest).

// Cells per unit of time: K / (l - f), or 0 when l - f is not positive and
// finite (every t strictly between f and l then falls in cell 0).
__device__ __forceinline__ float dir_scale(float f, float l, uint32_t K) {
    const float span = __fsub_rn(l, f);
    return span > 0.0f && span < __builtin_inff() ? __fdiv_rn(static_cast<float>(K), span) : 0.0f;
}

// The cell of time t, in [0, K); non-decreasing in t.
__device__ __forceinline__ uint32_t dir_cell(float t, float f, float l, float sc, uint32_t K) {
    if (!(t > f)) return 0;
    if (t >= l) return K - 1;
    const float x = __fmul_rn(__fsub_rn(t, f), sc);   // >= 0: t > f
    const uint32_t c = x < static_cast<float>(K) ? static_cast<uint32_t>(x) : K;
    return c < K - 1 ? c : K - 1;
}

}  // namespace tgl
