// Index build (Section 3.3; Appendix "Index build"): k-means over the keys of
// every (sequence, KV head) at once. The coarse problem clusters the
// directions u = k / ||k|| of R_b into n_list centers; each of the M subspace
// problems clusters the residual slices (u - c_a)^(m) into K codewords. One
// Lloyd iteration = the assignment (the encode pass of the update, run over
// all of R_b) + the kernels below:
//
//  * group_kernel: one workgroup per problem; a stable counting sort of the
//    problem's tokens by their center (LDS histogram, prefix sum, placement
//    chunk by chunk in token order), so that every mean below adds its
//    members in a fixed order.
//  * centers_kernel: one workgroup per (center, problem), groups of one
//    thread per dimension over the members; the float64 mean of the
//    members' directions, residual slices or values (the list means).
//  * reseed_kernel: one workgroup per problem; a center without members
//    takes the point farthest from its assigned center (farthest first, ties
//    to the smaller token id; one point per empty center, in center order).
//  * init_centers_kernel: the starting centers, the direction or residual
//    slice of caller-drawn tokens.
#include "device_common.h"
#include "pqhsa_internal.h"

namespace pqhsa {

constexpr int kGroupThreads = 1024;
constexpr int kGroupScanPer = kMaxLists / kGroupThreads;

struct Problem {
    int bg, m, nkeys, dims;
};

__device__ __forceinline__ Problem problem_of(const Dims& D, int kind, int p) {
    const int M = D.pq_bits == 4 ? Pq4::M : Pq8::M;
    const int K = D.pq_bits == 4 ? Pq4::K : Pq8::K;
    if (kind == 1) return Problem{p / M, p % M, K, kHeadDim / M};
    return Problem{p, 0, D.n_list, kHeadDim};
}

// the vector of token t for a problem: its direction (kind 0), the residual
// slice of subspace m (kind 1) or its value (kind 2), element x
template <typename T>
__device__ __forceinline__ float token_elem(const Dims& D, int kind, const KV& kv, int bg, int m,
                                            int dims, int t, int x, const int32_t* ids_tm,
                                            const float* norms_tm, const float* centroids) {
    const int b = bg / D.Hkv, g = bg % D.Hkv;
    const int64_t row = b * kv.sb + g * kv.sh + static_cast<int64_t>(t) * kv.sn;
    if (kind == 2) return load1<T>(static_cast<const T*>(kv.v) + row + x);
    const int col = m * dims + x;
    const float r = norms_tm[static_cast<int64_t>(bg) * D.rcap + t];
    const float u = r > 0.0f ? load1<T>(static_cast<const T*>(kv.k) + row + col) / r : 0.0f;
    if (kind == 0) return u;
    const int a = ids_tm[static_cast<int64_t>(bg) * D.rcap + t];
    return u - centroids[(static_cast<int64_t>(bg) * D.n_list + a) * kHeadDim + col];
}

__device__ __forceinline__ int64_t center_index(const Dims& D, int kind, const Problem& pr, int c,
                                                int x) {
    if (kind == 1) {
        const int M = kHeadDim / pr.dims;
        return ((static_cast<int64_t>(pr.bg) * M + pr.m) * pr.nkeys + c) * pr.dims + x;
    }
    return (static_cast<int64_t>(pr.bg) * D.n_list + c) * kHeadDim + x;
}

__global__ __launch_bounds__(kGroupThreads) void group_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                              int kind, const int32_t* ids_tm,
                                                              const uint8_t* codes_tm,
                                                              int32_t* order, int32_t* offs) {
    __shared__ int cnt[kMaxLists];
    __shared__ int placed[kMaxLists];
    __shared__ int chunk[kGroupThreads];
    __shared__ int wtot[kGroupThreads / kWave];
    const int p = blockIdx.x;
    const Problem pr = problem_of(D, kind, p);
    const int M = D.pq_bits == 4 ? Pq4::M : Pq8::M;
    const int b = pr.bg / D.Hkv;
    const int t0 = lo.v[b], t1 = hi.v[b];
    const int tid = threadIdx.x;
    const int64_t row = static_cast<int64_t>(pr.bg) * D.rcap;
    auto key = [&](int t) {
        return kind == 1 ? static_cast<int>(codes_tm[(row + t) * M + pr.m]) : ids_tm[row + t];
    };
    for (int j = tid; j < pr.nkeys; j += kGroupThreads) {
        cnt[j] = 0;
        placed[j] = 0;
    }
    __syncthreads();
    for (int t = t0 + tid; t < t1; t += kGroupThreads) atomicAdd(&cnt[key(t)], 1);
    __syncthreads();
    lds_exclusive_scan<kGroupThreads, kGroupScanPer>(cnt, pr.nkeys, wtot);
    int32_t* of = offs + static_cast<int64_t>(p) * (pr.nkeys + 1);
    for (int j = tid; j <= pr.nkeys; j += kGroupThreads) of[j] = j < pr.nkeys ? cnt[j] : t1 - t0;
    int32_t* ord = order + static_cast<int64_t>(p) * D.rcap;
    for (int c0 = t0; c0 < t1; c0 += kGroupThreads) {
        const int t = c0 + tid;
        const int j = t < t1 ? key(t) : -1;
        chunk[tid] = j;
        __syncthreads();
        if (t < t1) {
            int r = 0;
            for (int i = 0; i < tid; ++i) r += chunk[i] == j;
            ord[cnt[j] + placed[j] + r] = t;
        }
        __syncthreads();
        if (t < t1) atomicAdd(&placed[j], 1);
        __syncthreads();
    }
}

// 1024 threads per center: 1024 / dims groups of one thread per dimension;
// group gi adds members gi, gi + groups, ... in order, then group 0 adds the
// group sums in group order (a fixed order: the build is deterministic).
constexpr int kCenThreads = 1024;

template <typename T>
__global__ __launch_bounds__(kCenThreads) void centers_kernel(Dims D, int kind, KV kv,
                                                              const int32_t* ids_tm,
                                                              const float* norms_tm,
                                                              const float* centroids,
                                                              const int32_t* order,
                                                              const int32_t* offs, float* out) {
    __shared__ double part[kCenThreads];
    const int c = blockIdx.x;
    const int p = blockIdx.y;
    const Problem pr = problem_of(D, kind, p);
    if (c >= pr.nkeys) return;
    const int groups = kCenThreads / pr.dims;
    const int gi = threadIdx.x / pr.dims;
    const int x = threadIdx.x % pr.dims;
    const int32_t* of = offs + static_cast<int64_t>(p) * (pr.nkeys + 1);
    const int o0 = of[c], o1 = of[c + 1];
    if (o1 == o0) {   // empty: the list mean is 0; a center is re-seeded afterwards
        if (kind == 2 && gi == 0) out[center_index(D, kind, pr, c, x)] = 0.0f;
        return;
    }
    const int32_t* ord = order + static_cast<int64_t>(p) * D.rcap;
    double acc = 0.0;
#pragma unroll 4
    for (int i = o0 + gi; i < o1; i += groups)
        acc += static_cast<double>(
            token_elem<T>(D, kind, kv, pr.bg, pr.m, pr.dims, ord[i], x, ids_tm, norms_tm, centroids));
    part[threadIdx.x] = acc;
    __syncthreads();
    if (gi != 0) return;
    double sum = 0.0;
    for (int w = 0; w < groups; ++w) sum += part[w * pr.dims + x];
    out[center_index(D, kind, pr, c, x)] = static_cast<float>(sum / (o1 - o0));
}

template <typename T>
__global__ __launch_bounds__(kGroupThreads) void reseed_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                               int kind, KV kv,
                                                               const int32_t* ids_tm,
                                                               const float* norms_tm,
                                                               const float* centroids,
                                                               const int32_t* offs,
                                                               const float* dist_c,
                                                               const float* dist_f, float* out) {
    __shared__ int sof[kMaxLists + 1];
    __shared__ float wd[kGroupThreads / kWave];
    __shared__ int wt[kGroupThreads / kWave];
    __shared__ int pick;
    const int p = blockIdx.x;
    const Problem pr = problem_of(D, kind, p);
    const int M = D.pq_bits == 4 ? Pq4::M : Pq8::M;
    const int b = pr.bg / D.Hkv;
    const int t0 = lo.v[b], t1 = hi.v[b];
    const int tid = threadIdx.x;
    const int32_t* of = offs + static_cast<int64_t>(p) * (pr.nkeys + 1);
    for (int j = tid; j <= pr.nkeys; j += kGroupThreads) sof[j] = of[j];
    __syncthreads();
    const int64_t row = static_cast<int64_t>(pr.bg) * D.rcap;
    auto dist = [&](int t) { return kind == 1 ? dist_f[(row + t) * M + pr.m] : dist_c[row + t]; };
    float pd = __builtin_huge_valf();   // the previous pick: points must order after it
    int pt = -1;
    for (int c = 0; c < pr.nkeys; ++c) {
        if (sof[c + 1] != sof[c]) continue;   // uniform: every thread reads the same entry
        // the farthest point after (pd, pt) in the order (distance desc, token asc)
        float bd = -1.0f;
        int bt = -1;
        for (int t = t0 + tid; t < t1; t += kGroupThreads) {
            const float d = dist(t);
            const bool after = d < pd || (d == pd && t > pt);
            if (after && (d > bd || (d == bd && (bt < 0 || t < bt)))) {
                bd = d;
                bt = t;
            }
        }
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const float od = __shfl_xor(bd, off);
            const int ot = __shfl_xor(bt, off);
            if (ot >= 0 && (bt < 0 || od > bd || (od == bd && ot < bt))) {
                bd = od;
                bt = ot;
            }
        }
        if (lane_id() == 0) {
            wd[tid / kWave] = bd;
            wt[tid / kWave] = bt;
        }
        __syncthreads();
        if (tid == 0) {
            float d = -1.0f;
            int t = -1;
            for (int w = 0; w < kGroupThreads / kWave; ++w)
                if (wt[w] >= 0 && (t < 0 || wd[w] > d || (wd[w] == d && wt[w] < t))) {
                    d = wd[w];
                    t = wt[w];
                }
            pick = t;
            wd[0] = d;
        }
        __syncthreads();
        const int t = pick;
        const float d = wd[0];
        __syncthreads();
        if (t < 0) break;   // no point left
        if (tid < pr.dims)
            out[center_index(D, kind, pr, c, tid)] =
                token_elem<T>(D, kind, kv, pr.bg, pr.m, pr.dims, t, tid, ids_tm, norms_tm, centroids);
        pd = d;
        pt = t;
    }
}

template <typename T>
__global__ __launch_bounds__(kHeadDim) void init_centers_kernel(Dims D, int kind, KV kv,
                                                                const int32_t* init,
                                                                const int32_t* ids_tm,
                                                                const float* norms_tm,
                                                                const float* centroids,
                                                                float* out) {
    const int c = blockIdx.x;
    const int p = blockIdx.y;
    const Problem pr = problem_of(D, kind, p);
    const int x = threadIdx.x;
    if (c >= pr.nkeys || x >= pr.dims) return;
    const int t = init[static_cast<int64_t>(p) * pr.nkeys + c];
    out[center_index(D, kind, pr, c, x)] =
        token_elem<T>(D, kind, kv, pr.bg, pr.m, pr.dims, t, x, ids_tm, norms_tm, centroids);
}

static int n_problems(const Dims& D, int kind) {
    return D.B * D.Hkv * (kind == 1 ? (D.pq_bits == 4 ? Pq4::M : Pq8::M) : 1);
}
static int n_keys(const Dims& D, int kind) {
    return kind == 1 ? (D.pq_bits == 4 ? Pq4::K : Pq8::K) : D.n_list;
}

hipError_t launch_group(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                        const int32_t* ids_tm, const uint8_t* codes_tm, const BuildBufs& bb,
                        hipStream_t s) {
    hipLaunchKernelGGL(group_kernel, dim3(n_problems(D, kind)), dim3(kGroupThreads), 0, s, D, lo,
                       hi, kind, ids_tm, codes_tm, bb.order, bb.offs);
    return hipGetLastError();
}

hipError_t launch_centers(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                          const KV& kv, const int32_t* ids_tm, const float* norms_tm,
                          const float* centroids, const BuildBufs& bb, float* out, hipStream_t s) {
    (void)lo;
    (void)hi;
    const dim3 grid(n_keys(D, kind), n_problems(D, kind));
    if (kv.bf16)
        hipLaunchKernelGGL(centers_kernel<bf16_t>, grid, dim3(kCenThreads), 0, s, D, kind, kv, ids_tm,
                           norms_tm, centroids, bb.order, bb.offs, out);
    else
        hipLaunchKernelGGL(centers_kernel<float>, grid, dim3(kCenThreads), 0, s, D, kind, kv, ids_tm,
                           norms_tm, centroids, bb.order, bb.offs, out);
    return hipGetLastError();
}

hipError_t launch_reseed(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                         const KV& kv, const int32_t* ids_tm, const float* norms_tm,
                         const float* centroids, const BuildBufs& bb, float* out, hipStream_t s) {
    const dim3 grid(n_problems(D, kind));
    if (kv.bf16)
        hipLaunchKernelGGL(reseed_kernel<bf16_t>, grid, dim3(kGroupThreads), 0, s, D, lo, hi, kind,
                           kv, ids_tm, norms_tm, centroids, bb.offs, bb.dist_c, bb.dist_f, out);
    else
        hipLaunchKernelGGL(reseed_kernel<float>, grid, dim3(kGroupThreads), 0, s, D, lo, hi, kind,
                           kv, ids_tm, norms_tm, centroids, bb.offs, bb.dist_c, bb.dist_f, out);
    return hipGetLastError();
}

hipError_t launch_init_centers(const Dims& D, int kind, const KV& kv, const int32_t* init,
                               const int32_t* ids_tm, const float* norms_tm, const float* centroids,
                               float* out, hipStream_t s) {
    const dim3 grid(n_keys(D, kind), n_problems(D, kind));
    if (kv.bf16)
        hipLaunchKernelGGL(init_centers_kernel<bf16_t>, grid, dim3(kHeadDim), 0, s, D, kind, kv,
                           init, ids_tm, norms_tm, centroids, out);
    else
        hipLaunchKernelGGL(init_centers_kernel<float>, grid, dim3(kHeadDim), 0, s, D, kind, kv, init,
                           ids_tm, norms_tm, centroids, out);
    return hipGetLastError();
}

}  // namespace pqhsa
