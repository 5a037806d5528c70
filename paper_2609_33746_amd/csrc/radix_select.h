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
    int wave_aux[16];
};

// hist[digit] += 1 for every active lane. Lanes that share a digit are
// counted with one atomic (scores cluster, so the high digits of a pass are
// concentrated in a few bins and per-lane atomics would serialise on one LDS
// address); after two such rounds the remaining lanes add individually.
// Must be called by every lane of the wave.
__device__ __forceinline__ void hist_add(int* hist, uint32_t digit, bool active) {
    uint64_t todo = __ballot(active);
#pragma unroll
    for (int round = 0; round < 2; ++round) {
        if (todo == 0) return;
        const int leader = __ffsll(static_cast<long long>(todo)) - 1;
        const uint32_t d = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(digit), leader));
        const uint64_t same = __ballot(active && digit == d) & todo;
        if (lane_id() == leader) atomicAdd(&hist[d], __popcll(same));
        todo &= ~same;
    }
    if ((todo >> lane_id()) & 1ull) atomicAdd(&hist[digit], 1);
}

// All NT threads of the workgroup must call this with the same n and c,
// 1 <= c <= n.
template <int NT, typename KeyAt, typename Keep>
__device__ __forceinline__ SelectResult block_select_desc(KeyAt key_at, Keep keep, int n, int c,
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
        for (int i0 = 0; i0 < n; i0 += NT) {
            const int i = i0 + tid;
            bool act = false;
            uint32_t digit = 0u;
            if (i < n && keep(i)) {
                const uint32_t k = key_at(i);
                act = (k & pmask) == prefix;
                digit = (k >> shift) & 0xffu;
            }
            hist_add(sh.hist, digit, act);
        }
        __syncthreads();
        if (tid < kWave) {
            // lane l holds digits 255-4l .. 252-4l, i.e. descending order
            const int l = tid;
            int hv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) hv[j] = sh.hist[255 - 4 * l - j];
            const int mine = hv[0] + hv[1] + hv[2] + hv[3];
            const int incl = wave_incl_scan_i32(mine);
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
// (kReuse = false: the caller writes sh.wave_tot no more before its next
// barrier, so the trailing barrier that protects it is left out.)
template <int NT, bool kReuse = true>
__device__ __forceinline__ int block_excl_scan(int v, int& total, SelectScratch& sh) {
    constexpr int NW = NT / kWave;
    const int wave = threadIdx.x / kWave;
    const int incl = wave_incl_scan_i32(v);
    if (lane_id() == kWave - 1) sh.wave_tot[wave] = incl;
    __syncthreads();
    int wbase = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const int t = sh.wave_tot[i];
        wbase += i < wave ? t : 0;
        tot += t;
    }
    if constexpr (kReuse) __syncthreads();
    total = tot;
    return wbase + incl - v;
}

}  // namespace pqhsa
