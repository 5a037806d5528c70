// Workgroup helpers for order statistics over 32-bit order keys:
// min / max / count reductions, a shift-based histogram that is monotone in
// the key, and the search for the histogram bin holding the c-th largest key.
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

// Given hist[kHistBins], find the bin holding the c-th largest key (1-based);
// returns it and writes the number of keys in higher bins to `above`.
// All NT threads must call this; each owns kHistBins / NT bins.
template <int NT>
__device__ __forceinline__ int block_find_bin_desc(const int* hist, int c, int& above,
                                                   SelectScratch& ss, BlockScratch& bs) {
    constexpr int PER = kHistBins / NT;
    static_assert(PER * NT == kHistBins, "bins must divide evenly");
    const int t = threadIdx.x;
    int hv[PER];
    int mine = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        hv[j] = hist[kHistBins - 1 - (PER * t + j)];
        mine += hv[j];
    }
    int total = 0;
    int before = block_excl_scan<NT>(mine, total, ss);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        if (before < c && before + hv[j] >= c) {
            bs.bcast[0] = kHistBins - 1 - (PER * t + j);
            bs.bcast[1] = before;
        }
        before += hv[j];
    }
    __syncthreads();
    const int bin = bs.bcast[0];
    above = bs.bcast[1];
    __syncthreads();
    return bin;
}

}  // namespace pqhsa
