// Asymmetric-distance score of one indexed key (Eq. 2) from an LDS-resident
// lookup table. Used by the scan, the threshold sample, the re-scan path of
// the top-k stage and the debug score dump, so that all of them produce
// bit-identical approximate logits.
#pragma once

#include "device_common.h"
#include "pqhsa_internal.h"

namespace pqhsa {

// G consecutive floats of an LDS table entry.
template <int G>
__device__ __forceinline__ void load_entry(const float* e, float (&v)[G]) {
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
}

// Code z_m of subspace m from a position's code vector.
__device__ __forceinline__ uint32_t code_at(const uint4 c, int m) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    return (w[m >> 2] >> (8 * (m & 3))) & 0xffu;
}
__device__ __forceinline__ uint32_t code_at(const uint32_t c, int m) { return (c >> (4 * m)) & 0xfu; }

// LUT layout in LDS: [M][K][G] floats, entry (m, z, hh) = (q_hh^(m) . p_{m,z}) / sqrt(d)
// for the G query heads of one KV head (G = 1 for a single head's slice).
// fs[hh] = sum over m (in order m = 0..M-1) of the entries; the first entry
// initialises the sums (no 0 + x). With the table at a compile-time LDS
// address, each Pq8 entry address is one byte-select shift.
template <typename PQ, int G>
__device__ __forceinline__ void fine_sum(const float* __restrict__ lut, const typename PQ::Code c,
                                         float (&fs)[G]) {
#pragma unroll
    for (int m = 0; m < PQ::M; ++m) {
        float v[G];
        load_entry<G>(lut + (m * PQ::K + static_cast<int>(code_at(c, m))) * G, v);
#pragma unroll
        for (int hh = 0; hh < G; ++hh) fs[hh] = m == 0 ? v[hh] : fs[hh] + v[hh];
    }
}

// Pq4 tables are small enough to replicate: kRep4<G> copies of the [M][K][G]
// table interleaved entry by entry, entry (m, z) of copy c at floats
// ((m K + z) kRep4 + c) G, so that every entry spans 256 bytes of LDS. Lane l
// reads copy l mod kRep4, which puts the lanes of one LDS pass on distinct
// banks whatever their codes: the lookups are free of bank conflicts.
template <int G>
constexpr int kRep4 = 256 / (4 * G);
constexpr int kRep4Floats = Pq4::LUT_ROW * 64;   // one replicated table: 32 KB for any G

template <int G>
__device__ __forceinline__ void fine_sum_rep4(const float* __restrict__ lut_rep, uint32_t c,
                                              float (&fs)[G]) {
    const float* base = lut_rep + (lane_id() % kRep4<G>) * G;
#pragma unroll
    for (int m = 0; m < Pq4::M; ++m) {
        float v[G];
        load_entry<G>(base + (m * Pq4::K + static_cast<int>(code_at(c, m))) * 64, v);
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
template <typename PQ, int NT>
__device__ __forceinline__ void stage_head_lut(float* __restrict__ dst,
                                               const float* __restrict__ group_lut, int G,
                                               int hh) {
    for (int i = threadIdx.x; i < PQ::LUT_ROW; i += NT) dst[i] = group_lut[i * G + hh];
}

}  // namespace pqhsa
