// Workgroup-wide radix select over 32-bit order keys (8 bits per pass, most
// significant first): finds the c-th largest key of n keys and the number of
// keys strictly above it. Keys are read through a functor so that the same
// code serves LDS and global arrays.
#pragma once

#include "device_common.h"

namespace pqhsa {

struct SelectResult {
    uint32_t key;      // the c-th largest key
    int count_above;   // number of keys strictly greater than `key`
    int count_equal;   // number of keys equal to `key`
};

struct SelectScratch {
    int hist[256];
    int bcast[4];
    int wave_tot[16];
};

// All NT threads of the workgroup must call this with the same n and c,
// 1 <= c <= n.
template <int NT, typename KeyAt, typename Keep>
__device__ SelectResult block_select_desc(KeyAt key_at, Keep keep, int n, int c,
                                          SelectScratch& sh) {
    static_assert(NT >= 64, "needs at least one full wave");
    const int tid = threadIdx.x;
    uint32_t prefix = 0u, pmask = 0u;
    int remaining = c;
    int above_total = 0;
    int equal = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += NT) sh.hist[i] = 0;
        __syncthreads();
        for (int i = tid; i < n; i += NT) {
            if (!keep(i)) continue;
            const uint32_t k = key_at(i);
            if ((k & pmask) == prefix) atomicAdd(&sh.hist[(k >> shift) & 0xffu], 1);
        }
        __syncthreads();
        if (tid < kWave) {
            // lane l holds digits 255-4l .. 252-4l, i.e. descending order
            const int l = tid;
            int hv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) hv[j] = sh.hist[255 - 4 * l - j];
            const int mine = hv[0] + hv[1] + hv[2] + hv[3];
            int incl = mine;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const int t = __shfl_up(incl, off);
                if (l >= off) incl += t;
            }
            int before = incl - mine;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (before < remaining && before + hv[j] >= remaining) {
                    sh.bcast[0] = 255 - 4 * l - j;
                    sh.bcast[1] = before;
                    sh.bcast[2] = hv[j];
                }
                before += hv[j];
            }
        }
        __syncthreads();
        const int digit = sh.bcast[0];
        const int above = sh.bcast[1];
        equal = sh.bcast[2];
        remaining -= above;
        above_total += above;
        prefix |= static_cast<uint32_t>(digit) << shift;
        pmask |= 0xffu << shift;
        __syncthreads();
    }
    return {prefix, above_total, equal};
}

// Exclusive prefix of a per-thread count over the workgroup (NT threads);
// returns this thread's offset, writes the total to `total`.
template <int NT>
__device__ int block_excl_scan(int v, int& total, SelectScratch& sh) {
    constexpr int NW = NT / kWave;
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    int incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int t = __shfl_up(incl, off);
        if (lane >= off) incl += t;
    }
    if (lane == kWave - 1) sh.wave_tot[wave] = incl;
    __syncthreads();
    int wbase = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const int t = sh.wave_tot[i];
        if (i < wave) wbase += t;
        tot += t;
    }
    __syncthreads();
    total = tot;
    return wbase + incl - v;
}

}  // namespace pqhsa
