// Code scan (Section 3.1, Eq. 2; Section 3.3 "code scan with a fused per-list
// reduction"). Every indexed token of every list is scored for the G query
// heads that share its KV head, in one pass over the list-major uint8 codes.
//
// Work decomposition: the list-major positions of each (batch element, KV
// head) are cut into sub-chunks of kSub positions; one wave owns one
// sub-chunk, and a workgroup holds kScanWaves consecutive sub-chunks of the
// same KV head so that they share one copy of the group LUT in LDS. Each wave
// keeps the metadata of the lists it walks (start offsets, first segment,
// coarse terms) in a 64-lane register window, so the inner loop issues no
// dependent global loads.
//
// Per token and head the wave computes l~ and then either
//   * emits (l~, list id and position) as a top-k candidate when
//     l~ >= tau_lo (the sampled threshold of its row), compacted in position
//     order at the start of the sub-chunk's own region of the row's candidate
//     buffer, or
//   * adds exp(l~ - tau_lo) (< 1) to the running mass of its inverted list.
// Tokens below tau_lo can never be in the top-k (tau_lo <= the k-th largest
// score whenever at least k candidates exist), so these masses are exactly
// the "below threshold" part of M_j in Eq. 4; the unselected candidates are
// added by the top-k stage. Masses are written per (list, sub-chunk)
// segment, so no atomics are used and the result does not depend on
// scheduling.
#include "device_common.h"
#include "pq_score.h"
#include "pqhsa_internal.h"

namespace pqhsa {

// Metadata of lists [base, base + 63) held one list per lane; lane l also
// holds the start of list base + l, so list base + i spans
// [start(i), start(i + 1)).
template <int G>
struct ListWindow {
    int base;
    int start;
    int seg;
    float cf[G];

    __device__ __forceinline__ void load(const int32_t* loff, const int32_t* seg0,
                                         const float* coarse, int n_list, int first) {
        base = first;
        const int j = first + lane_id();
        start = j <= n_list ? loff[j] : 0x7fffffff;
        seg = j < n_list ? seg0[j] : 0;
#pragma unroll
        for (int hh = 0; hh < G; ++hh) cf[hh] = j < n_list ? coarse[j * G + hh] : 0.0f;
    }
    __device__ __forceinline__ int start_of(int i) const { return __builtin_amdgcn_readlane(start, i); }
    __device__ __forceinline__ int seg_of(int i) const { return __builtin_amdgcn_readlane(seg, i); }
    __device__ __forceinline__ float cf_of(int hh, int i) const {
        return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cf[hh]), i));
    }
};
constexpr int kWindowLists = kWave - 1;

template <int G>
__device__ __forceinline__ void flush_segment(const Dims& D, const Work& w, int bg, int seg,
                                              float (&acc)[G]) {
    float mine = 0.0f;
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        const float tot = wave_sum(acc[hh]);
        if (lane_id() == hh) mine = tot;
        acc[hh] = 0.0f;
    }
    if (lane_id() < G) w.seg_sum[(static_cast<int64_t>(bg) * D.nseg_cap + seg) * G + lane_id()] = mine;
}

template <int G>
__global__ __launch_bounds__(kScanWaves * kWave) void scan_kernel(Dims D, Index ix, Work w,
                                                                  const ScanWG* __restrict__ table) {
    extern __shared__ float lut_s[];   // [M][K][G]
    const ScanWG& entry = table[blockIdx.x];
    const int bg = entry.bg;
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;

    const int n_r = ix.n_r[b];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int sc = entry.sub0 + wave;
    const bool active = sc * kSub < n_r;
    const int p_begin = sc * kSub;
    const int p_end = min(p_begin + kSub, n_r);
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const uint4* codes = reinterpret_cast<const uint4*>(ix.codes) + base;
    const int32_t* loff = ix.loff + static_cast<int64_t>(bg) * (D.n_list + 1);
    const int32_t* seg0 = ix.seg0 + static_cast<int64_t>(bg) * (D.n_list + 1);
    const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * G;
    const int row0 = b * D.Hq + g * G;

    // issue this wave's code, norm and list-metadata loads before staging the LUT
    constexpr int kIters = kSub / kWave;
    uint4 c_pre[kIters];
    float r_pre[kIters];
#pragma unroll
    for (int it = 0; it < kIters; ++it) {
        const int p = p_begin + it * kWave + lane;
        c_pre[it] = make_uint4(0u, 0u, 0u, 0u);
        r_pre[it] = 0.0f;
        if (active && p < p_end) {
            c_pre[it] = codes[p];
            r_pre[it] = ix.norms[base + p];
        }
    }
    ListWindow<G> win;
    win.load(loff, seg0, coarse, D.n_list, active ? entry.list0[wave] : 0);
    float tlo[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) tlo[hh] = w.tau_lo[row0 + hh];
    {
        const float4* src = reinterpret_cast<const float4*>(w.lut + static_cast<int64_t>(bg) * kLutRow * G);
        float4* dst = reinterpret_cast<float4*>(lut_s);
        for (int i = threadIdx.x; i < kLutRow * G / 4; i += kScanWaves * kWave) dst[i] = src[i];
    }
    __syncthreads();
    if (!active) return;

    int ci = 0;   // window index of the current list
    int cur_start = win.start_of(0);
    int cur_end = win.start_of(1);
    float acc[G];
    int cbase[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) { acc[hh] = 0.0f; cbase[hh] = 0; }

#pragma unroll
    for (int it = 0; it < kIters; ++it) {
        const int p_first = p_begin + it * kWave;
        if (p_first >= p_end) break;
        const int p = p_first + lane;
        const bool valid = p < p_end;
        const int p_last = min(p_first + kWave - 1, p_end - 1);
        float fs[G];
        fine_sum<G>(lut_s, c_pre[it], fs);
        const float r = r_pre[it];
        float s[G];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) s[hh] = 0.0f;
        int my_list = 0;

        // walk the lists that cover [p_first, p_last] (wave-uniform)
        while (true) {
            const bool in = valid && p >= cur_start && p < cur_end;
            if (in) my_list = win.base + ci;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                const float sc_h = pq_logit(r, win.cf_of(hh, ci), fs[hh]);
                if (in) s[hh] = sc_h;
                acc[hh] += (in && sc_h < tlo[hh]) ? __expf(sc_h - tlo[hh]) : 0.0f;
            }
            if (cur_end > p_last) break;
            flush_segment<G>(D, w, bg, win.seg_of(ci) + (sc - cur_start / kSub), acc);
            do {
                ++ci;
                if (ci == kWindowLists) {
                    win.load(loff, seg0, coarse, D.n_list, win.base + kWindowLists);
                    ci = 0;
                }
                cur_start = cur_end;
                cur_end = win.start_of(ci + 1);
            } while (cur_end == cur_start);
        }

        // candidates >= tau_lo, compacted in position order
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            const bool pred = valid && s[hh] >= tlo[hh];
            const uint64_t mask = __ballot(pred);
            if (pred) {
                const int64_t o = static_cast<int64_t>(row0 + hh) * D.rcap + p_begin + cbase[hh] +
                                  lanes_below(mask);
                w.cand_score[o] = s[hh];
                w.cand_pos[o] = static_cast<int32_t>((static_cast<uint32_t>(my_list) << kPosBits) |
                                                     static_cast<uint32_t>(p));
            }
            cbase[hh] += __popcll(mask);
        }
    }
    flush_segment<G>(D, w, bg, win.seg_of(ci) + (sc - cur_start / kSub), acc);
    int mine = 0;
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
        if (lane == hh) mine = cbase[hh];
    if (lane < G) w.cand_cnt[static_cast<int64_t>(row0 + lane) * D.nsub_cap + sc] = mine;
}

template <int G>
static hipError_t launch_scan_t(const Dims& D, const Index& ix, const Work& w, const ScanWG* table,
                                int n_wg, hipStream_t s) {
    const size_t lds = static_cast<size_t>(kLutRow) * G * sizeof(float);
    hipLaunchKernelGGL((scan_kernel<G>), dim3(n_wg), dim3(kScanWaves * kWave), lds, s, D, ix, w,
                       table);
    return hipGetLastError();
}

hipError_t configure_scan() {
    // the G = 8 group LUT (128 KB) exceeds the default dynamic LDS limit
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&scan_kernel<8>),
                               hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(kLutRow * 8 * sizeof(float)));
}

hipError_t launch_scan(const Dims& D, const Index& ix, const Work& w, const ScanWG* table, int n_wg,
                       hipStream_t s) {
    if (n_wg == 0) return hipSuccess;
    switch (D.G) {
        case 1: return launch_scan_t<1>(D, ix, w, table, n_wg, s);
        case 2: return launch_scan_t<2>(D, ix, w, table, n_wg, s);
        case 4: return launch_scan_t<4>(D, ix, w, table, n_wg, s);
        case 8: return launch_scan_t<8>(D, ix, w, table, n_wg, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace pqhsa
