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

// The same stable grouping for problems of at most kGroupFastKeys centers,
// spread over many workgroups and without the O(chunk^2) rank. A problem's
// tokens are cut into segments of kSegTok; three launches:
//  * group_count_kernel, one workgroup per (segment, problem): the
//    segment's key counts (LDS atomics) to seg_hist[problem][segment][key];
//  * group_scan_kernel, one workgroup per problem: the centers' offsets
//    (key-major, then segment order: a stable layout), and each segment's
//    first position per key in place of its counts;
//  * group_place_kernel, one workgroup per (segment, problem): wave w owns
//    the w-th sixteenth of the segment; the per-wave counts turn into each
//    wave's first position per key, and each wave places its tokens 64 at a
//    time, the rank among equal keys of a step coming from one ballot per
//    distinct key and its base from one LDS atomic of the key's first lane.
constexpr int kGroupWaves = kGroupThreads / kWave;
constexpr int kGroupFastKeys = 1024;
constexpr int kSegTok = kBuildSegTok;   // tokens per segment

__device__ __forceinline__ int group_key(const Dims& D, int kind, const Problem& pr, int64_t row, int t,
                                         const int32_t* ids_tm, const uint8_t* codes_tm) {
    const int M = D.pq_bits == 4 ? Pq4::M : Pq8::M;
    const int k = kind == 1 ? static_cast<int>(codes_tm[(row + t) * M + pr.m]) : ids_tm[row + t];
    return min(max(k, 0), pr.nkeys - 1);
}

__global__ __launch_bounds__(kGroupThreads) void group_count_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                                    int kind, const int32_t* ids_tm,
                                                                    const uint8_t* codes_tm,
                                                                    int32_t* seg_hist, int nseg) {
    __shared__ int hist[kGroupFastKeys];
    const int seg = blockIdx.x, p = blockIdx.y;
    const Problem pr = problem_of(D, kind, p);
    const int b = pr.bg / D.Hkv;
    const int s0 = lo.v[b] + seg * kSegTok, s1 = min(s0 + kSegTok, hi.v[b]);
    const int64_t row = static_cast<int64_t>(pr.bg) * D.rcap;
    for (int j = threadIdx.x; j < pr.nkeys; j += kGroupThreads) hist[j] = 0;
    __syncthreads();
    for (int t = s0 + static_cast<int>(threadIdx.x); t < s1; t += kGroupThreads)
        atomicAdd(&hist[group_key(D, kind, pr, row, t, ids_tm, codes_tm)], 1);
    __syncthreads();
    int32_t* out = seg_hist + (static_cast<int64_t>(p) * nseg + seg) * pr.nkeys;
    for (int j = threadIdx.x; j < pr.nkeys; j += kGroupThreads) out[j] = hist[j];
}

__global__ __launch_bounds__(kGroupThreads) void group_scan_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                                   int kind, int32_t* seg_hist, int nseg,
                                                                   int32_t* offs) {
    __shared__ int tot[kGroupFastKeys];
    __shared__ int wtot[kGroupWaves];
    const int p = blockIdx.x;
    const Problem pr = problem_of(D, kind, p);
    const int b = pr.bg / D.Hkv;
    const int nk = pr.nkeys;
    int32_t* h = seg_hist + static_cast<int64_t>(p) * nseg * nk;
    for (int j = threadIdx.x; j < nk; j += kGroupThreads) {
        int sum = 0;
        for (int sg = 0; sg < nseg; ++sg) sum += h[static_cast<int64_t>(sg) * nk + j];
        tot[j] = sum;
    }
    __syncthreads();
    lds_exclusive_scan<kGroupThreads, 1>(tot, nk, wtot);
    int32_t* of = offs + static_cast<int64_t>(p) * (nk + 1);
    for (int j = threadIdx.x; j <= nk; j += kGroupThreads) of[j] = j < nk ? tot[j] : hi.v[b] - lo.v[b];
    for (int j = threadIdx.x; j < nk; j += kGroupThreads) {
        int at = tot[j];
        for (int sg = 0; sg < nseg; ++sg) {
            const int64_t i = static_cast<int64_t>(sg) * nk + j;
            const int c = h[i];
            h[i] = at;
            at += c;
        }
    }
}

__global__ __launch_bounds__(kGroupThreads) void group_place_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                                    int kind, const int32_t* ids_tm,
                                                                    const uint8_t* codes_tm,
                                                                    const int32_t* seg_hist, int nseg,
                                                                    int32_t* order) {
    __shared__ int hist[kGroupWaves][kGroupFastKeys];
    const int seg = blockIdx.x, p = blockIdx.y;
    const Problem pr = problem_of(D, kind, p);
    const int b = pr.bg / D.Hkv;
    const int s0 = lo.v[b] + seg * kSegTok, s1 = min(s0 + kSegTok, hi.v[b]);
    if (s0 >= s1) return;
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = lane_id();
    const int nk = pr.nkeys;
    const int64_t row = static_cast<int64_t>(pr.bg) * D.rcap;
    // the wave's part of the segment
    const int n = s1 - s0;
    const int per = (n + kGroupWaves - 1) / kGroupWaves;
    const int w0 = s0 + min(wave * per, n), w1 = s0 + min(wave * per + per, n);
    for (int i = tid; i < kGroupWaves * kGroupFastKeys; i += kGroupThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    for (int t = w0 + lane; t < w1; t += kWave) atomicAdd(&hist[wave][group_key(D, kind, pr, row, t, ids_tm, codes_tm)], 1);
    __syncthreads();
    const int32_t* base_g = seg_hist + (static_cast<int64_t>(p) * nseg + seg) * nk;
    for (int j = tid; j < nk; j += kGroupThreads) {
        int at = base_g[j];
#pragma unroll
        for (int w = 0; w < kGroupWaves; ++w) {
            const int c = hist[w][j];
            hist[w][j] = at;
            at += c;
        }
    }
    __syncthreads();
    int32_t* ord = order + static_cast<int64_t>(p) * D.rcap;
    for (int c0 = w0; c0 < w1; c0 += kWave) {
        const int t = c0 + lane;
        const bool valid = t < w1;
        const int k = valid ? group_key(D, kind, pr, row, t, ids_tm, codes_tm) : 0;
        // ranks among equal keys from ballots alone (registers), then one LDS
        // atomic per distinct key, made by the key's first lane
        uint64_t todo = __ballot(valid);
        int leader_of = lane, rank = 0, cnt = 0;
        while (todo) {
            const int leader = __ffsll(static_cast<long long>(todo)) - 1;
            const int kl = __builtin_amdgcn_readlane(k, leader);
            const uint64_t same = __ballot(valid && k == kl) & todo;
            if ((same >> lane) & 1ull) {
                leader_of = leader;
                rank = lanes_below(same);
            }
            if (lane == leader) cnt = __popcll(same);
            todo &= ~same;
        }
        int base = 0;
        if (valid && lane == leader_of) base = atomicAdd(&hist[wave][k], cnt);
        base = __shfl(base, leader_of);
        if (valid) ord[base + rank] = t;
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

hipError_t launch_group_segments(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                                 const int32_t* ids_tm, const uint8_t* codes_tm, int32_t* seg_hist,
                                 int32_t* order, int32_t* offs, hipStream_t s) {
    int max_n = 0;
    for (int b = 0; b < D.B; ++b) max_n = hi.v[b] - lo.v[b] > max_n ? hi.v[b] - lo.v[b] : max_n;
    const int nseg = (max_n + kSegTok - 1) / kSegTok;
    const dim3 grid(nseg, n_problems(D, kind));
    if (nseg > 0) {
        hipLaunchKernelGGL(group_count_kernel, grid, dim3(kGroupThreads), 0, s, D, lo, hi, kind, ids_tm,
                           codes_tm, seg_hist, nseg);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // also with no tokens: the offsets are written
    hipLaunchKernelGGL(group_scan_kernel, dim3(n_problems(D, kind)), dim3(kGroupThreads), 0, s, D, lo,
                       hi, kind, seg_hist, nseg, offs);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || nseg == 0) return e;
    hipLaunchKernelGGL(group_place_kernel, grid, dim3(kGroupThreads), 0, s, D, lo, hi, kind, ids_tm,
                       codes_tm, seg_hist, nseg, order);
    return hipGetLastError();
}

hipError_t launch_group(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                        const int32_t* ids_tm, const uint8_t* codes_tm, const BuildBufs& bb,
                        hipStream_t s) {
    if (n_keys(D, kind) <= kGroupFastKeys && bb.seg_hist)
        return launch_group_segments(D, lo, hi, kind, ids_tm, codes_tm, bb.seg_hist, bb.order, bb.offs, s);
    else
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

// ---------------------------------------------------------------------------
// assign_kernel: the coarse assignment of the build on the matrix cores.
// ||u - c||^2 = ||u||^2 + ||c||^2 - 2 u . c, and the dot products of a tile
// of tokens with a chunk of centers are one fp32 matrix product: 128 tokens
// per workgroup (4 waves x 2 tiles of 16), centers in chunks of 64 (4 tiles
// of 16), K = 128 dimensions as 32 steps of v_mfma_f32_16x16x4f32. In step
// j, lane group q (lane / 16) contributes dimension 32 q + j, so each lane
// reads 32 contiguous floats of its row; rows are 132 floats apart in LDS,
// which puts the 16 rows of a read on distinct 16-byte bank groups. Every
// lane keeps a running (distance, center) minimum for the 2 token columns
// it holds, over the 4 centers of each tile it sees; the 4 lane groups are
// folded at the end, ties going to the smaller center id. The directions,
// norms and distances are fp32; the distance of the chosen center is
// written for the re-seeding.
// ---------------------------------------------------------------------------
constexpr int kAsgThreads = 256;
constexpr int kAsgTok = 128;                  // tokens per workgroup
constexpr int kAsgCen = 64;                   // centers per chunk
constexpr int kAsgLd = kHeadDim + 4;          // LDS row stride (floats)
static_assert(kAsgTok * kAsgLd >= 2 * kAsgCen * kAsgLd, "the token rows hold a center chunk");

typedef float asg_v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void asg_fold(float& d, int& i, float od, int oi) {
    if (od < d || (od == d && oi < i)) {
        d = od;
        i = oi;
    }
}

template <typename T>
__global__ __launch_bounds__(kAsgThreads) void assign_kernel(Dims D, BatchInts lo, BatchInts hi, KV kv,
                                                             const float* __restrict__ centroids,
                                                             int32_t* __restrict__ ids_tm,
                                                             float* __restrict__ dist_c) {
    __shared__ float4 rows4[kAsgTok * kAsgLd / 4];   // token rows, then center chunks
    __shared__ float cn[kAsgCen];                    // ||c||^2 of the chunk's centers
    __shared__ float un[kAsgTok];                    // ||u||^2 of the tokens
    float* rows = reinterpret_cast<float*>(rows4);
    const int b = blockIdx.z;
    const int g = blockIdx.y;
    const int t_base = lo.v[b] + static_cast<int>(blockIdx.x) * kAsgTok;
    if (t_base >= hi.v[b]) return;
    const int nt = min(kAsgTok, hi.v[b] - t_base);
    const int bg = b * D.Hkv + g;
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = lane_id();
    const int col = lane % 16;   // the lane's token column (B) / center row (A) in a tile
    const int q = lane / 16;     // its lane group: dimensions 32 q .. 32 q + 31

    // 1) the directions u = k / ||k|| of the workgroup's tokens into LDS:
    //    16 threads per token, 8 dimensions each
    const T* kb = static_cast<const T*>(kv.k) + b * kv.sb + g * kv.sh;
#pragma unroll
    for (int it = 0; it < kAsgTok / 16; ++it) {
        const int tk = it * 16 + tid / 16;
        const int x0 = (tid % 16) * 8;
        float x[8];
        if (tk < nt) {
            Load8<T>::run(kb + static_cast<int64_t>(t_base + tk) * kv.sn + x0, x);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = 0.0f;
        }
        float ss = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) ss = fmaf(x[e], x[e], ss);
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) ss += __shfl_xor(ss, off);
        const float r = sqrtf(ss);
        float uu = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            x[e] = r > 0.0f ? x[e] / r : 0.0f;
            uu = fmaf(x[e], x[e], uu);
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) uu += __shfl_xor(uu, off);
        if (tid % 16 == 0) un[tk] = uu;
        float4* dst = reinterpret_cast<float4*>(rows + tk * kAsgLd + x0);
        dst[0] = make_float4(x[0], x[1], x[2], x[3]);
        dst[1] = make_float4(x[4], x[5], x[6], x[7]);
    }
    __syncthreads();
    // 2) the B operands: token rows (2 tiles of the wave), 32 dimensions each
    float bv[2][32];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
        const float4* src = reinterpret_cast<const float4*>(rows + (wave * 32 + tt * 16 + col) * kAsgLd + 32 * q);
#pragma unroll
        for (int v = 0; v < 8; ++v) {
            const float4 f = src[v];
            bv[tt][4 * v] = f.x; bv[tt][4 * v + 1] = f.y; bv[tt][4 * v + 2] = f.z; bv[tt][4 * v + 3] = f.w;
        }
    }
    float best_d[2] = {__builtin_huge_valf(), __builtin_huge_valf()};
    int best_i[2] = {0, 0};   // a valid id even if every distance is NaN

    // 3) the centers, a chunk of 64 at a time
    const float* cen = centroids + static_cast<int64_t>(bg) * D.n_list * kHeadDim;
    for (int c0 = 0; c0 < D.n_list; c0 += kAsgCen) {
        __syncthreads();   // the previous chunk (or the token rows) is no longer read
#pragma unroll
        for (int it = 0; it < kAsgCen * kHeadDim / 4 / kAsgThreads; ++it) {
            const int idx = it * kAsgThreads + tid;
            const int ci = idx / 32;          // 32 float4 per center row
            const int p = idx % 32;
            const bool ok = c0 + ci < D.n_list;
            const float4 v = ok ? reinterpret_cast<const float4*>(cen + static_cast<int64_t>(c0 + ci) * kHeadDim)[p]
                                : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            float ss = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
#pragma unroll
            for (int off = 1; off < 32; off <<= 1) ss += __shfl_xor(ss, off);
            if (p == 0) cn[ci] = ss;
            reinterpret_cast<float4*>(rows + ci * kAsgLd)[p] = v;
        }
        __syncthreads();
        // dot products: 4 center tiles x 2 token tiles, 8 independent chains
        asg_v4f acc[4][2];
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) acc[ct][tt] = asg_v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int j4 = 0; j4 < 8; ++j4) {
            float4 av[4];
#pragma unroll
            for (int ct = 0; ct < 4; ++ct)
                av[ct] = reinterpret_cast<const float4*>(rows + (ct * 16 + col) * kAsgLd + 32 * q)[j4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                for (int ct = 0; ct < 4; ++ct) {
                    const float a = jj == 0 ? av[ct].x : jj == 1 ? av[ct].y : jj == 2 ? av[ct].z : av[ct].w;
#pragma unroll
                    for (int tt = 0; tt < 2; ++tt)
                        acc[ct][tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[tt][4 * j4 + jj],
                                                                        acc[ct][tt], 0, 0, 0);
                }
        }
        // distances up to ||u||^2: row 4 q + i of tile ct is center c0 + 16 ct + 4 q + i
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int cl = ct * 16 + 4 * q + i;
                if (c0 + cl < D.n_list) {
                    const float c2 = cn[cl];
#pragma unroll
                    for (int tt = 0; tt < 2; ++tt)
                        asg_fold(best_d[tt], best_i[tt], fmaf(-2.0f, acc[ct][tt][i], c2), c0 + cl);
                }
            }
    }
    // 4) the 4 lane groups of a token column, then the outputs
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
        for (int off = 16; off < kWave; off <<= 1) {
            const float od = __shfl_xor(best_d[tt], off);
            const int oi = __shfl_xor(best_i[tt], off);
            asg_fold(best_d[tt], best_i[tt], od, oi);
        }
        const int tk = wave * 32 + tt * 16 + col;
        if (q == 0 && tk < nt) {
            const int64_t at = static_cast<int64_t>(bg) * D.rcap + t_base + tk;
            ids_tm[at] = best_i[tt];
            if (dist_c) dist_c[at] = fmaxf(best_d[tt] + un[tk], 0.0f);
        }
    }
}

// ---------------------------------------------------------------------------
// subspace_kernel: the codeword search of the build on the matrix cores, for
// tokens whose lists are known (ids_tm): the residual r = u - c_a of each
// token, then per subspace m the nearest codeword by ||p||^2 - 2 r^(m) . p
// (16x16x4 fp32 MFMA tiles: 16 codewords x 16 tokens, DSUB / 4 steps). Lane
// group q contributes dimensions m DSUB + q DSUB / 4 + s of subspace m in
// step s, so its operands are contiguous. Writes the norms ||k||, the codes
// and the chosen squared distances (dist_f, or null); ties go to the smaller
// codeword.
// ---------------------------------------------------------------------------
template <typename PQ>
constexpr int kSubRound = PQ::K >= 256 ? 4 : PQ::M;   // subspaces per LDS round
template <typename PQ>
constexpr int kSubLd = PQ::DSUB + 1;                   // codeword row stride (odd: distinct banks)
static_assert(kSubRound<Pq8> * Pq8::K * kSubLd<Pq8> <= kAsgTok * kAsgLd, "codewords fit the token rows");
static_assert(kSubRound<Pq4> * Pq4::K * kSubLd<Pq4> <= kAsgTok * kAsgLd, "codewords fit the token rows");

template <typename T, typename PQ>
__global__ __launch_bounds__(kAsgThreads) void subspace_kernel(
    Dims D, BatchInts lo, BatchInts hi, KV kv, const float* __restrict__ centroids,
    const float* __restrict__ codebooks, const int32_t* __restrict__ ids_tm,
    uint8_t* __restrict__ codes_tm, float* __restrict__ norms_tm, float* __restrict__ dist_f) {
    constexpr int M = PQ::M, K = PQ::K, DS = PQ::DSUB, S = DS / 4, SR = kSubRound<PQ>, LD = kSubLd<PQ>;
    constexpr int NCT = K / 16;   // codeword tiles per subspace
    static_assert(K % 16 == 0 && DS % 4 == 0 && M % SR == 0, "tiling");
    __shared__ float4 rows4[kAsgTok * kAsgLd / 4];   // residual rows, then codewords
    __shared__ float pn[SR * K];                     // ||p||^2 of the round's codewords
    float* rows = reinterpret_cast<float*>(rows4);
    const int b = blockIdx.z;
    const int g = blockIdx.y;
    const int t_base = lo.v[b] + static_cast<int>(blockIdx.x) * kAsgTok;
    if (t_base >= hi.v[b]) return;
    const int nt = min(kAsgTok, hi.v[b] - t_base);
    const int bg = b * D.Hkv + g;
    const int64_t row0 = static_cast<int64_t>(bg) * D.rcap + t_base;
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = lane_id();
    const int col = lane % 16;
    const int q = lane / 16;

    // 1) residuals u - c_a into LDS, 16 threads per token (8 dimensions each);
    //    the norms ||k|| out
    const T* kb = static_cast<const T*>(kv.k) + b * kv.sb + g * kv.sh;
    const float* cen = centroids + static_cast<int64_t>(bg) * D.n_list * kHeadDim;
#pragma unroll
    for (int it = 0; it < kAsgTok / 16; ++it) {
        const int tk = it * 16 + tid / 16;
        const int x0 = (tid % 16) * 8;
        float x[8];
        int a = 0;
        if (tk < nt) {
            Load8<T>::run(kb + static_cast<int64_t>(t_base + tk) * kv.sn + x0, x);
            a = min(max(ids_tm[row0 + tk], 0), D.n_list - 1);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = 0.0f;
        }
        float ss = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) ss = fmaf(x[e], x[e], ss);
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) ss += __shfl_xor(ss, off);
        const float r = sqrtf(ss);
        if (tid % 16 == 0 && tk < nt) norms_tm[row0 + tk] = r;
        const float4* cp = reinterpret_cast<const float4*>(cen + static_cast<int64_t>(a) * kHeadDim + x0);
        const float4 c0 = cp[0], c1 = cp[1];
        const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = tk < nt ? (r > 0.0f ? x[e] / r : 0.0f) - cv[e] : 0.0f;
        float4* dst = reinterpret_cast<float4*>(rows + tk * kAsgLd + x0);
        dst[0] = make_float4(x[0], x[1], x[2], x[3]);
        dst[1] = make_float4(x[4], x[5], x[6], x[7]);
    }
    __syncthreads();
    // 2) the B operands: lane (col, q) of token tile tt holds dimensions
    //    m DS + q S + s of its token, for every m and s
    float bv[2][M * S];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
        const float* src = rows + (wave * 32 + tt * 16 + col) * kAsgLd;
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int s2 = 0; s2 < S; ++s2) bv[tt][m * S + s2] = src[m * DS + q * S + s2];
    }

    // 3) the subspaces, SR at a time through LDS
    const float* cb = codebooks + static_cast<int64_t>(bg) * M * K * DS;
#pragma unroll
    for (int m0 = 0; m0 < M; m0 += SR) {   // unrolled: bv is indexed by m
        __syncthreads();   // the residual rows or the previous round are no longer read
        for (int i = tid; i < SR * K * DS; i += kAsgThreads) {
            const int z = i / DS, x = i % DS;   // z over the round's SR * K codewords
            rows[z * LD + x] = cb[static_cast<int64_t>(m0) * K * DS + i];
        }
        __syncthreads();
        for (int z = tid; z < SR * K; z += kAsgThreads) {
            float ss = 0.0f;
#pragma unroll
            for (int x = 0; x < DS; ++x) ss = fmaf(rows[z * LD + x], rows[z * LD + x], ss);
            pn[z] = ss;
        }
        __syncthreads();
#pragma unroll
        for (int mm = 0; mm < SR; ++mm) {
            const int m = m0 + mm;
            float best_d[2] = {__builtin_huge_valf(), __builtin_huge_valf()};
            int best_z[2] = {0, 0};
#pragma unroll 4
            for (int ct = 0; ct < NCT; ++ct) {
                const float* arow = rows + (mm * K + ct * 16 + col) * LD + q * S;
                asg_v4f acc[2] = {asg_v4f{0.0f, 0.0f, 0.0f, 0.0f}, asg_v4f{0.0f, 0.0f, 0.0f, 0.0f}};
#pragma unroll
                for (int s2 = 0; s2 < S; ++s2) {
                    const float a = arow[s2];
#pragma unroll
                    for (int tt = 0; tt < 2; ++tt)
                        acc[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[tt][m * S + s2], acc[tt], 0, 0, 0);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int zl = ct * 16 + 4 * q + i;   // codeword of row 4 q + i
                    const float p2 = pn[mm * K + zl];
#pragma unroll
                    for (int tt = 0; tt < 2; ++tt) asg_fold(best_d[tt], best_z[tt], fmaf(-2.0f, acc[tt][i], p2), zl);
                }
            }
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) {
                float r2 = 0.0f;   // ||r^(m)||^2 of the lane's token, over the 4 lane groups
#pragma unroll
                for (int s2 = 0; s2 < S; ++s2) r2 = fmaf(bv[tt][m * S + s2], bv[tt][m * S + s2], r2);
#pragma unroll
                for (int off = 16; off < kWave; off <<= 1) {
                    r2 += __shfl_xor(r2, off);
                    const float od = __shfl_xor(best_d[tt], off);
                    const int oz = __shfl_xor(best_z[tt], off);
                    asg_fold(best_d[tt], best_z[tt], od, oz);
                }
                const int tk = wave * 32 + tt * 16 + col;
                if (q == 0 && tk < nt) {
                    codes_tm[(row0 + tk) * M + m] = static_cast<uint8_t>(best_z[tt]);
                    if (dist_f) dist_f[(row0 + tk) * M + m] = fmaxf(best_d[tt] + r2, 0.0f);
                }
            }
        }
    }
}

hipError_t launch_subspace(const Dims& D, const BatchInts& lo, const BatchInts& hi, int max_n,
                           const KV& kv, const float* centroids, const float* codebooks,
                           const int32_t* ids_tm, uint8_t* codes_tm, float* norms_tm, float* dist_f,
                           hipStream_t s) {
    if (max_n <= 0) return hipSuccess;
    const dim3 grid((max_n + kAsgTok - 1) / kAsgTok, D.Hkv, D.B);
#define PQHSA_SUB(TT, PQT)                                                                      \
    hipLaunchKernelGGL((subspace_kernel<TT, PQT>), grid, dim3(kAsgThreads), 0, s, D, lo, hi, kv, \
                       centroids, codebooks, ids_tm, codes_tm, norms_tm, dist_f)
    if (kv.bf16) {
        if (D.pq_bits == 4) PQHSA_SUB(bf16_t, Pq4); else PQHSA_SUB(bf16_t, Pq8);
    } else {
        if (D.pq_bits == 4) PQHSA_SUB(float, Pq4); else PQHSA_SUB(float, Pq8);
    }
#undef PQHSA_SUB
    return hipGetLastError();
}

hipError_t launch_assign(const Dims& D, const BatchInts& lo, const BatchInts& hi, int max_n,
                         const KV& kv, const float* centroids, int32_t* ids_tm, float* dist_c,
                         hipStream_t s) {
    if (max_n <= 0) return hipSuccess;
    const dim3 grid((max_n + kAsgTok - 1) / kAsgTok, D.Hkv, D.B);
    if (kv.bf16)
        hipLaunchKernelGGL(assign_kernel<bf16_t>, grid, dim3(kAsgThreads), 0, s, D, lo, hi, kv,
                           centroids, ids_tm, dist_c);
    else
        hipLaunchKernelGGL(assign_kernel<float>, grid, dim3(kAsgThreads), 0, s, D, lo, hi, kv,
                           centroids, ids_tm, dist_c);
    return hipGetLastError();
}

}  // namespace pqhsa
