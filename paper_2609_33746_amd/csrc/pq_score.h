// Asymmetric-distance score of one indexed key (Eq. 2) from an LDS-resident
// lookup table. Used by the scan, the threshold sample, the re-scan path of
// the top-k stage and the debug score dump, so that all of them produce
// bit-identical approximate logits.
#pragma once

#include "device_common.h"
#include "pqhsa_internal.h"

namespace pqhsa {

// LUT layout in LDS: [M][K][G] floats, entry (m, z, hh) = (q_hh^(m) . p_{m,z}) / sqrt(d)
// for the G query heads of one KV head. `stride` is G for the group LUT or 1 for a
// single head's slice. fs[hh] = sum over m (in order m = 0..M-1) of the entries.
// The first entry initialises the sums (no 0 + x). With the table at a
// compile-time LDS address, each entry address is one byte-select shift.
template <int G>
__device__ __forceinline__ void fine_sum(const float* __restrict__ lut, const uint4 c,
                                         float (&fs)[G]) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
    for (int m = 0; m < kPqM; ++m) {
        const uint32_t z = (w[m >> 2] >> (8 * (m & 3))) & 0xffu;
        const float* e = lut + (m * kKsub + static_cast<int>(z)) * G;
        float v[G];
        if constexpr (G == 8) {
            const float4 a = *reinterpret_cast<const float4*>(e);
            const float4 b = *reinterpret_cast<const float4*>(e + 4);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else if constexpr (G == 4) {
            const float4 a = *reinterpret_cast<const float4*>(e);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        } else if constexpr (G == 2) {
            const float2 a = *reinterpret_cast<const float2*>(e);
            v[0] = a.x; v[1] = a.y;
        } else {
            v[0] = e[0];
        }
#pragma unroll
        for (int hh = 0; hh < G; ++hh) fs[hh] = m == 0 ? v[hh] : fs[hh] + v[hh];
    }
}

// l~ = r_i * (coarse + fine sum); the 1/sqrt(d) and r_q factors of Eq. 2 are
// already folded into the tables (they hold q/sqrt(d) products).
__device__ __forceinline__ float pq_logit(float r, float coarse, float fs) {
    return r * (coarse + fs);
}

// Copy one query head's slice (hh of G) of the group LUT into LDS [M][K].
template <int NT>
__device__ __forceinline__ void stage_head_lut(float* __restrict__ dst,
                                               const float* __restrict__ group_lut, int G,
                                               int hh) {
    for (int i = threadIdx.x; i < kLutRow; i += NT) dst[i] = group_lut[i * G + hh];
}

}  // namespace pqhsa
