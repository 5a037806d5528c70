// Index preparation (list-major reorder of codes and norms) and the
// diagnostics of pqhsa_decode_debug.
#include "device_common.h"
#include "pq_score.h"
#include "pqhsa_internal.h"

namespace pqhsa {

// Codes of one position from the caller's one-byte-per-code layout: Pq8 as
// is (16 bytes), Pq4 packed two per byte (code m in bits 4m .. 4m + 3; the
// caller's codes are < 16, only their low four bits are kept).
__device__ __forceinline__ uint4 prepared_code(const uint8_t* p, Pq8) {
    return *reinterpret_cast<const uint4*>(p);
}
__device__ __forceinline__ uint32_t prepared_code(const uint8_t* p, Pq4) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    uint32_t out = 0u;
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const uint32_t byte = ((m < 4 ? v.x : v.y) >> (8 * (m & 3))) & 0xfu;
        out |= byte << (4 * m);
    }
    return out;
}

// codes_out[bg][pos] = codes_in[bg][perm[pos]] (prepared layout), same for norms.
template <typename PQ>
__global__ __launch_bounds__(256) void gather_index_kernel(Dims D, const uint8_t* __restrict__ codes_in,
                                                           const float* __restrict__ norms_in,
                                                           Index ix,
                                                           typename PQ::Code* __restrict__ codes_out,
                                                           float* __restrict__ norms_out) {
    const int bg = blockIdx.y;
    const int b = bg / D.Hkv;
    const int pos = blockIdx.x * 256 + threadIdx.x;
    if (pos >= ix.n_r[b]) return;
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const int tok = ix.perm[base + pos];
    codes_out[base + pos] = prepared_code(codes_in + (base + tok) * PQ::M, PQ{});
    norms_out[base + pos] = norms_in[base + tok];
}

hipError_t launch_prepare_gather(const Dims& D, const uint8_t* codes_in, const float* norms_in,
                                 const Index& ix, uint8_t* codes_out, float* norms_out,
                                 hipStream_t s) {
    dim3 grid((D.rcap + 255) / 256, D.B * D.Hkv);
    if (D.pq_bits == 4)
        hipLaunchKernelGGL(gather_index_kernel<Pq4>, grid, dim3(256), 0, s, D, codes_in, norms_in,
                           ix, reinterpret_cast<uint32_t*>(codes_out), norms_out);
    else
        hipLaunchKernelGGL(gather_index_kernel<Pq8>, grid, dim3(256), 0, s, D, codes_in, norms_in,
                           ix, reinterpret_cast<uint4*>(codes_out), norms_out);
    return hipGetLastError();
}

// The threshold sample of each (b, kv head): sample slot s takes the code,
// norm and list id of list-major position sample_position(s) (slot data of
// positions past the sample are those of position 0, never used).
template <typename PQ>
__global__ __launch_bounds__(256) void sample_slab_kernel(Dims D, Index ix,
                                                          typename PQ::Code* __restrict__ codes_out,
                                                          float* __restrict__ norms_out,
                                                          int32_t* __restrict__ list_out) {
    const int bg = blockIdx.x;
    const int b = bg / D.Hkv;
    const int n_r = ix.n_r[b];
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const typename PQ::Code* codes = reinterpret_cast<const typename PQ::Code*>(ix.codes) + base;
    const SampleRuns sr = sample_runs(max(n_r, 1));
    for (int sl = threadIdx.x; sl < kMaxSamples; sl += 256) {
        int pos = 0;
        if (n_r == 0 || !sample_position(sr, sl, n_r, pos)) pos = 0;
        const int64_t o = static_cast<int64_t>(bg) * kMaxSamples + sl;
        codes_out[o] = codes[pos];
        norms_out[o] = ix.norms[base + pos];
        list_out[o] = static_cast<int32_t>(ix.pos_word[base + pos] >> kPosBits);
    }
}

hipError_t launch_sample_slab(const Dims& D, const Index& ix, uint8_t* samp_codes, float* samp_norms,
                              int32_t* samp_list, hipStream_t s) {
    if (D.pq_bits == 4)
        hipLaunchKernelGGL(sample_slab_kernel<Pq4>, dim3(D.B * D.Hkv), dim3(256), 0, s, D, ix,
                           reinterpret_cast<uint32_t*>(samp_codes), samp_norms, samp_list);
    else
        hipLaunchKernelGGL(sample_slab_kernel<Pq8>, dim3(D.B * D.Hkv), dim3(256), 0, s, D, ix,
                           reinterpret_cast<uint4*>(samp_codes), samp_norms, samp_list);
    return hipGetLastError();
}

// Global value mean over R_b per (b, g) for variant C (Appendix B): the list
// means weighted by the list sizes, sum_j |R_j| v_bar_j / |R_b| (0 for an
// empty R_b), accumulated in float64. Workgroup (b g, dimension chunk):
// kGlobGroups groups of one thread per dimension of the chunk take every
// kGlobGroups-th list, then group 0 adds the group sums in a fixed order.
constexpr int kGlobDims = 32;                       // dimensions per workgroup
constexpr int kGlobGroups = 1024 / kGlobDims;       // list groups per workgroup

__global__ __launch_bounds__(1024) void glob_mean_kernel(Dims D, Index ix, float* glob) {
    __shared__ double part[kGlobGroups][kGlobDims];
    const int bg = blockIdx.x;
    const int b = bg / D.Hkv;
    const int t = blockIdx.y * kGlobDims + threadIdx.x % kGlobDims;
    const int gi = threadIdx.x / kGlobDims;
    const int32_t* loff = ix.loff + static_cast<int64_t>(bg) * (D.n_list + 1);
    const float* means = ix.means + static_cast<int64_t>(bg) * D.n_list * kHeadDim + t;
    double acc = 0.0;
#pragma unroll 8
    for (int j = gi; j < D.n_list; j += kGlobGroups)
        acc += static_cast<double>(loff[j + 1] - loff[j]) * static_cast<double>(means[j * kHeadDim]);
    part[gi][threadIdx.x % kGlobDims] = acc;
    __syncthreads();
    if (gi != 0) return;
    for (int g = 1; g < kGlobGroups; ++g) acc += part[g][threadIdx.x];
    const int n_r = ix.n_r[b];
    glob[static_cast<int64_t>(bg) * kHeadDim + t] = n_r > 0 ? static_cast<float>(acc / n_r) : 0.0f;
}

hipError_t launch_glob_mean(const Dims& D, const Index& ix, float* glob, hipStream_t s) {
    hipLaunchKernelGGL(glob_mean_kernel, dim3(D.B * D.Hkv, kHeadDim / kGlobDims), dim3(1024), 0, s,
                       D, ix, glob);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// diagnostics
// ---------------------------------------------------------------------------
constexpr int kDbgThreads = 256;
constexpr int kSortCap = 8192;   // largest k whose selected set the debug call can sort

__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

// Approximate logit of every indexed token, scattered by token id.
template <typename PQ>
__global__ __launch_bounds__(kDbgThreads) void score_dump_kernel(Dims D, Index ix, Work w,
                                                                 float* __restrict__ scores,
                                                                 int64_t out_stride) {
    __shared__ float lut_s[PQ::LUT_ROW];
    const int row = blockIdx.y;
    const int b = row / D.Hq;
    const int h = row % D.Hq;
    const int g = h / D.G;
    const int hh = h % D.G;
    const int bg = b * D.Hkv + g;
    stage_head_lut<PQ, kDbgThreads>(lut_s, w.lut + static_cast<int64_t>(bg) * PQ::LUT_ROW * D.G,
                                    D.G, hh);
    __syncthreads();
    const int n_r = ix.n_r[b];
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const typename PQ::Code* codes = reinterpret_cast<const typename PQ::Code*>(ix.codes) + base;
    const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * D.G;
    for (int pos = blockIdx.x * kDbgThreads + threadIdx.x; pos < n_r;
         pos += gridDim.x * kDbgThreads) {
        float fs[1];
        fine_sum<PQ, 1>(lut_s, codes[pos], fs);
        const uint32_t wd = ix.pos_word[base + pos];
        const float s = pq_logit(ix.norms[base + pos], coarse[(wd >> kPosBits) * D.G + hh], fs[0]);
        scores[row * out_stride + (wd & kPosMask)] = s;
    }
}

// Sort the selected token ids of each row ascending (bitonic, in LDS), pad with -1,
// and count |B n R_j| = |R_j| - |T n R_j| per list.
__global__ __launch_bounds__(kDbgThreads) void sel_debug_kernel(Dims D, BatchArgs ba, Index ix,
                                                                Work w, int32_t* __restrict__ selected,
                                                                int32_t* __restrict__ unselected) {
    __shared__ int keys[kSortCap];
    __shared__ int counts[kMaxLists];
    const int row = blockIdx.x;
    const int b = row / D.Hq;
    const int g = (row % D.Hq) / D.G;
    const int bg = b * D.Hkv + g;
    const int k = ba.topk[b];
    const int32_t* st = w.sel_tok + static_cast<int64_t>(row) * D.max_topk;
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    // the selected token ids, sorted (both outputs use them)
    int n2 = 1;
    while (n2 < k) n2 <<= 1;
    for (int i = threadIdx.x; i < n2; i += kDbgThreads) keys[i] = i < k ? st[i] : 0x7fffffff;
    __syncthreads();
    for (int size = 2; size <= n2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = threadIdx.x; i < n2; i += kDbgThreads) {
                const int j = i ^ stride;
                if (j > i) {
                    const bool up = (i & size) == 0;
                    const int a = keys[i], c = keys[j];
                    if ((a > c) == up) {
                        keys[i] = c;
                        keys[j] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    if (selected) {
        int32_t* out = selected + static_cast<int64_t>(row) * D.max_topk;
        for (int i = threadIdx.x; i < D.max_topk; i += kDbgThreads) out[i] = i < k ? keys[i] : -1;
    }
    if (unselected) {
        // a position is selected when its token id is among the sorted keys
        const int32_t* loff = ix.loff + static_cast<int64_t>(bg) * (D.n_list + 1);
        for (int j = threadIdx.x; j < D.n_list; j += kDbgThreads) counts[j] = loff[j + 1] - loff[j];
        __syncthreads();
        const int n_r = ba.n_r[b];
        for (int pos = threadIdx.x; pos < n_r; pos += kDbgThreads) {
            const uint32_t wd = ix.pos_word[base + pos];
            const int tok = static_cast<int>(wd & kPosMask);
            int lo = 0, hi = k;   // first key >= tok
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (keys[mid] < tok) lo = mid + 1;
                else hi = mid;
            }
            if (lo < k && keys[lo] == tok) atomicSub(&counts[wd >> kPosBits], 1);
        }
        __syncthreads();
        int32_t* out = unselected + static_cast<int64_t>(row) * D.n_list;
        for (int j = threadIdx.x; j < D.n_list; j += kDbgThreads) out[j] = counts[j];
    }
}

hipError_t launch_debug(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                        int32_t* selected, int32_t* unselected, float* scores, hipStream_t s) {
    if (scores) {
        const int64_t n = static_cast<int64_t>(D.B) * D.Hq * D.rcap;
        hipLaunchKernelGGL(fill_f32_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0,
                           s, scores, n, __builtin_nanf(""));
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        dim3 grid(64, D.B * D.Hq);
        if (D.pq_bits == 4)
            hipLaunchKernelGGL(score_dump_kernel<Pq4>, grid, dim3(kDbgThreads), 0, s, D, ix, w,
                               scores, static_cast<int64_t>(D.rcap));
        else
            hipLaunchKernelGGL(score_dump_kernel<Pq8>, grid, dim3(kDbgThreads), 0, s, D, ix, w,
                               scores, static_cast<int64_t>(D.rcap));
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (selected || unselected) {
        hipLaunchKernelGGL(sel_debug_kernel, dim3(D.B * D.Hq), dim3(kDbgThreads), 0, s, D, ba, ix, w,
                           selected, unselected);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace pqhsa
