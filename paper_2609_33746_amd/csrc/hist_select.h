// Workgroup helpers for order statistics over 32-bit order keys:
// min / max / count reductions, a shift-based histogram that is monotone in
// the key, and the search (by one wave) for the histogram bin holding the c-th
// largest key.
#pragma once

#include "device_common.h"
#include "radix_select.h"

namespace pqhsa {

constexpr int kHistBins = 2048;

struct BlockScratch {
    uint32_t v[16][3];
    int bcast[4];
};

// Reduce (min, max, count) over the workgroup; every thread gets the result.
template <int NT>
__device__ __forceinline__ void block_min_max_count(uint32_t& mn, uint32_t& mx, uint32_t& cnt,
                                                    BlockScratch& s) {
    constexpr int NW = NT / kWave;
    const int wave = threadIdx.x / kWave;
    mn = wave_min_u32(mn);
    mx = wave_max_u32(mx);
    cnt = wave_sum_u32(cnt);
    if (lane_id() == 0) {
        s.v[wave][0] = mn;
        s.v[wave][1] = mx;
        s.v[wave][2] = cnt;
    }
    __syncthreads();
    mn = s.v[0][0];
    mx = s.v[0][1];
    cnt = s.v[0][2];
#pragma unroll
    for (int i = 1; i < NW; ++i) {
        mn = min(mn, s.v[i][0]);
        mx = max(mx, s.v[i][1]);
        cnt += s.v[i][2];
    }
    __syncthreads();
}

// Right shift that maps [kmin, kmax] onto at most kHistBins bins:
// bin(key) = (key - kmin) >> shift is non-decreasing in key.
__device__ __forceinline__ int bin_shift(uint32_t kmin, uint32_t kmax) {
    const uint32_t range = kmax - kmin;
    const int bits = range == 0 ? 0 : 32 - __clz(static_cast<int>(range));
    return bits > 11 ? bits - 11 : 0;
}

// The histogram bin holding the c-th largest entry (1 <= c <= the count in
// hist), found by one wave; `above` receives the entries in higher bins.
// Lane l sums the 32 bins of rank 32 l .. 32 l + 31 from the top (read in a
// lane-rotated order, so the lanes of one read hit distinct LDS banks), a
// wave scan finds the lane whose bins reach c, and a second scan over that
// lane's 32 bins, one per lane, finds the bin.
__device__ __forceinline__ int wave_find_bin_desc(const int* hist, int c, int& above) {
    constexpr int PER = kHistBins / kWave;
    static_assert(PER == 32, "two scans of 32 bins");
    const int lane = lane_id();
    int sum = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) sum += hist[kHistBins - 1 - (PER * lane + ((q + lane) & (PER - 1)))];
    const int incl = wave_incl_scan_i32(sum);
    const uint64_t r1 = __ballot(incl >= c);
    const int L = r1 ? __ffsll(static_cast<long long>(r1)) - 1 : kWave - 1;
    const int before = __builtin_amdgcn_readlane(incl - sum, L);
    const int v = lane < PER ? hist[kHistBins - 1 - (PER * L + lane)] : 0;
    const int incl2 = wave_incl_scan_i32(v);
    const uint64_t r2 = __ballot(lane < PER && before + incl2 >= c);
    const int M = r2 ? __ffsll(static_cast<long long>(r2)) - 1 : PER - 1;
    above = before + __builtin_amdgcn_readlane(incl2 - v, M);
    return kHistBins - 1 - (PER * L + M);
}

}  // namespace pqhsa
