// Incremental index update (Section 3.3): tokens that leave the local window
// are encoded into the existing lists, without re-clustering, and the list
// means are refreshed over the grown lists.
//
//  * encode_one_kernel, one token per workgroup (updates of a few hundred
//    tokens; the build's passes over all of R use the matrix-core search in
//    the build's source): the key is split into
//    its norm r and direction u (Section 3.1); u goes to the list with the
//    nearest centroid, and each slice of the residual u - c_a to its nearest
//    codeword. Squared Euclidean distances in fp32; ties go to the smaller
//    list id or codeword index. Writes the token-major list id, codes (one
//    code per byte) and norm.
//  * means_update_kernel, after the merge below: one workgroup per (list,
//    kv head, sequence) adds the new members' values to the list's float64
//    value sum and writes the mean v_bar' = sum / (n_old + n_new) in fp32. The
//    sums start at |R_j| v_bar_j when an index is prepared or built, so the
//    fp32 means never feed back into later updates and do not drift.
//
// The list-major layout is then merged on the device (update_lists_kernel,
// shift_positions_kernel below) and codes and norms gathered into it.
#include "device_common.h"
#include "pqhsa_internal.h"

namespace pqhsa {

constexpr int kEncThreads = 256;

// (d, i) < (od, oi) lexicographically: the smaller distance, then the smaller index
__device__ __forceinline__ void argmin_fold(float& d, int& i, float od, int oi) {
    if (od < d || (od == d && oi < i)) {
        d = od;
        i = oi;
    }
}

// argmin over the 64 lanes of a wave by (distance, id)
__device__ __forceinline__ void wave_argmin64(float& d, int& i) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const float od = __shfl_xor(d, off);
        const int oi = __shfl_xor(i, off);
        argmin_fold(d, i, od, oi);
    }
}

// One workgroup per token: for updates of a few hundred tokens, where
// 64-token tiles would leave most of the chip idle. The same choices as
// the build's search up to fp32 rounding order.
template <typename T, typename PQ>
__global__ __launch_bounds__(kEncThreads) void encode_one_kernel(
    Dims D, BatchInts lo, BatchInts hi, const T* __restrict__ kcache, int64_t sb, int64_t sh,
    int64_t sn, const float* __restrict__ centroids, const float* __restrict__ codebooks,
    int32_t* __restrict__ ids_tm, uint8_t* __restrict__ codes_tm, float* __restrict__ norms_tm) {
    __shared__ float su[kHeadDim];           // u, then the residual u - c_a
    __shared__ float sdist[kMaxLists];       // coarse distances, then [M][K] fine ones
    __shared__ float wsum[kEncThreads / kWave];
    __shared__ int sa;
    static_assert(PQ::M * PQ::K <= kMaxLists, "fine distances fit the coarse buffer");
    const int b = blockIdx.z;
    const int g = blockIdx.y;
    const int t = lo.v[b] + static_cast<int>(blockIdx.x);
    if (t >= hi.v[b]) return;
    const int bg = b * D.Hkv + g;
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = lane_id();

    // r = ||k||, u = k / r (u = 0 for a zero key)
    float kx = 0.0f;
    if (tid < kHeadDim) kx = load1<T>(kcache + b * sb + g * sh + t * sn + tid);
    float ss = kx * kx;
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    if (lane == 0) wsum[wave] = ss;
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int w = 0; w < kEncThreads / kWave; ++w) tot += wsum[w];
    const float r = sqrtf(tot);
    if (tid < kHeadDim) su[tid] = r > 0.0f ? kx / r : 0.0f;
    __syncthreads();

    // nearest centroid
    const float* cen = centroids + static_cast<int64_t>(bg) * D.n_list * kHeadDim;
    for (int j = tid; j < D.n_list; j += kEncThreads) {
        const float4* c4 = reinterpret_cast<const float4*>(cen + static_cast<int64_t>(j) * kHeadDim);
        float acc = 0.0f;
#pragma unroll 8
        for (int x = 0; x < kHeadDim / 4; ++x) {
            const float4 c = c4[x];
            const float d0 = su[4 * x] - c.x, d1 = su[4 * x + 1] - c.y;
            const float d2 = su[4 * x + 2] - c.z, d3 = su[4 * x + 3] - c.w;
            acc = fmaf(d0, d0, acc);
            acc = fmaf(d1, d1, acc);
            acc = fmaf(d2, d2, acc);
            acc = fmaf(d3, d3, acc);
        }
        sdist[j] = acc;
    }
    __syncthreads();
    if (wave == 0) {
        float bd = __builtin_huge_valf();
        int bi = 0;   // a valid id even if every distance is NaN
        for (int j = lane; j < D.n_list; j += kWave) argmin_fold(bd, bi, sdist[j], j);
        wave_argmin64(bd, bi);
        if (lane == 0) sa = bi;
    }
    __syncthreads();
    const int a = sa;
    if (tid < kHeadDim) su[tid] -= cen[static_cast<int64_t>(a) * kHeadDim + tid];
    __syncthreads();

    // nearest codeword of every subspace slice of the residual
    const float* cb = codebooks + static_cast<int64_t>(bg) * PQ::M * PQ::K * PQ::DSUB;
    for (int p = tid; p < PQ::M * PQ::K; p += kEncThreads) {
        const int m = p / PQ::K;
        float acc = 0.0f;
#pragma unroll
        for (int x = 0; x < PQ::DSUB; ++x) {
            const float dx = su[m * PQ::DSUB + x] - cb[static_cast<int64_t>(p) * PQ::DSUB + x];
            acc = fmaf(dx, dx, acc);
        }
        sdist[p] = acc;
    }
    __syncthreads();
    const int64_t tok = static_cast<int64_t>(bg) * D.rcap + t;
    for (int m = wave; m < PQ::M; m += kEncThreads / kWave) {
        float bd = __builtin_huge_valf();
        int bi = 0;   // a valid id even if every distance is NaN
        for (int z = lane; z < PQ::K; z += kWave) argmin_fold(bd, bi, sdist[m * PQ::K + z], z);
        wave_argmin64(bd, bi);
        if (lane == 0) codes_tm[tok * PQ::M + m] = static_cast<uint8_t>(bi);
    }
    if (tid == 0) {
        ids_tm[tok] = a;
        norms_tm[tok] = r;
    }
}

// One workgroup per (list j, kv head g, sequence b), one thread per dimension,
// after the merge: the list's new members are the last (new size - old size)
// positions of its new range, in token order.
template <typename T>
__global__ __launch_bounds__(kHeadDim) void means_update_kernel(
    Dims D, const T* __restrict__ vcache, int64_t sb, int64_t sh, int64_t sn,
    const int32_t* __restrict__ old_loff, const int32_t* __restrict__ new_loff,
    const int32_t* __restrict__ perm_new, float* __restrict__ means, double* __restrict__ sums) {
    const int j = blockIdx.x;
    const int g = blockIdx.y;
    const int b = blockIdx.z;
    const int bg = b * D.Hkv + g;
    const int64_t lo = static_cast<int64_t>(bg) * (D.n_list + 1) + j;
    const int n_old = old_loff[lo + 1] - old_loff[lo];
    const int end = new_loff[lo + 1];
    const int n_all = end - new_loff[lo];
    if (n_all == n_old) return;
    const int x = threadIdx.x;
    const int32_t* perm = perm_new + static_cast<int64_t>(bg) * D.rcap;
    const T* vb = vcache + b * sb + g * sh + x;
    const int64_t at = (static_cast<int64_t>(bg) * D.n_list + j) * kHeadDim + x;
    double s = sums[at];
    for (int p = end - (n_all - n_old); p < end; ++p)
        s += static_cast<double>(load1<T>(vb + static_cast<int64_t>(perm[p]) * sn));
    sums[at] = s;
    means[at] = static_cast<float>(s / static_cast<double>(n_all));
}

// The float64 value sums of the lists from the means of a prepared or built
// index: sum_j = |R_j| v_bar_j (0 for an empty list).
__global__ __launch_bounds__(kHeadDim) void init_sums_kernel(Dims D, const int32_t* __restrict__ loff,
                                                             const float* __restrict__ means,
                                                             double* __restrict__ sums) {
    const int j = blockIdx.x;
    const int bg = blockIdx.y;
    const int64_t lo = static_cast<int64_t>(bg) * (D.n_list + 1) + j;
    const int64_t at = (static_cast<int64_t>(bg) * D.n_list + j) * kHeadDim + threadIdx.x;
    sums[at] = static_cast<double>(loff[lo + 1] - loff[lo]) * static_cast<double>(means[at]);
}

hipError_t launch_init_sums(const Dims& D, const int32_t* loff, const float* means, double* sums,
                            hipStream_t s) {
    hipLaunchKernelGGL(init_sums_kernel, dim3(D.n_list, D.B * D.Hkv), dim3(kHeadDim), 0, s, D, loff,
                       means, sums);
    return hipGetLastError();
}

// List-major rebuild after an update, on the device. The new tokens of a
// (b, g) have larger ids than every indexed one, so each list keeps its old
// members in order and appends its new ones in increasing id: an old position
// p of list j moves to p + (new members of lists before j), and the r-th new
// member of list j lands at old_end(j) + (new members of lists before j) + r.
//
// update_lists_kernel: one workgroup per (b, g). Counts the new members per
// list (LDS atomics), scans the counts into the per-list shifts, writes the
// new list offsets, and places the new tokens chunk by chunk in id order
// (rank within a chunk = earlier lanes of the chunk with the same list).
constexpr int kListThreads = 1024;
constexpr int kScanPer = kMaxLists / kListThreads;   // list counts per thread in the scan

__global__ __launch_bounds__(kListThreads) void update_lists_kernel(
    Dims D, BatchInts lo, BatchInts hi, const int32_t* __restrict__ ids_tm,
    const int32_t* __restrict__ old_loff, int32_t* __restrict__ new_loff,
    int32_t* __restrict__ shift, int32_t* __restrict__ perm_new, uint32_t* __restrict__ pos_new,
    int32_t* __restrict__ n_r_dev, int32_t* __restrict__ n_seq_dev) {
    __shared__ int cnt[kMaxLists];     // new members per list, then the exclusive scan
    __shared__ int placed[kMaxLists];  // new members placed so far per list
    __shared__ int chunk[kListThreads];
    __shared__ int wtot[kListThreads / kWave];
    const int bg = blockIdx.x;
    const int b = bg / D.Hkv;
    const int tid = threadIdx.x;
    const int L = D.n_list;
    const int t0 = lo.v[b], t1 = hi.v[b];
    if (tid == 0 && bg % D.Hkv == 0) {
        n_r_dev[b] = t1 - D.n_sink;
        n_seq_dev[b] = t1 + D.n_local;
    }
    for (int j = tid; j < L; j += kListThreads) {
        cnt[j] = 0;
        placed[j] = 0;
    }
    __syncthreads();
    const int32_t* ids = ids_tm + static_cast<int64_t>(bg) * D.rcap;
    // list ids are clamped into [0, n_list): a prepare checks them separately
    // (check_ids_kernel) and fails the call, so an invalid id never indexes LDS
    auto list_of = [&](int t) { return min(max(ids[t], 0), L - 1); };
    for (int t = t0 + tid; t < t1; t += kListThreads) atomicAdd(&cnt[list_of(t)], 1);
    __syncthreads();
    lds_exclusive_scan<kListThreads, kScanPer>(cnt, L, wtot);
    const int32_t* ol = old_loff + static_cast<int64_t>(bg) * (L + 1);
    int32_t* nl = new_loff + static_cast<int64_t>(bg) * (L + 1);
    for (int j = tid; j <= L; j += kListThreads) nl[j] = ol[j] + (j < L ? cnt[j] : t1 - t0);
    for (int j = tid; j < L; j += kListThreads) shift[static_cast<int64_t>(bg) * L + j] = cnt[j];
    const int64_t row = static_cast<int64_t>(bg) * D.rcap;
    for (int c0 = t0; c0 < t1; c0 += kListThreads) {
        const int t = c0 + tid;
        const int j = t < t1 ? list_of(t) : -1;
        chunk[tid] = j;
        __syncthreads();
        if (t < t1) {
            int r = 0;
            for (int i = 0; i < tid; ++i) r += chunk[i] == j;
            const int pos = ol[j + 1] + cnt[j] + placed[j] + r;
            perm_new[row + pos] = t;
            pos_new[row + pos] = (static_cast<uint32_t>(j) << kPosBits) | static_cast<uint32_t>(t);
        }
        __syncthreads();
        if (t < t1) atomicAdd(&placed[j], 1);
        __syncthreads();
    }
}

// shift_positions_kernel: the old members move right by their list's shift;
// positions past the new |R_b| are cleared (perm -1).
__global__ __launch_bounds__(256) void shift_positions_kernel(
    Dims D, BatchInts lo, BatchInts hi, const int32_t* __restrict__ shift,
    const int32_t* __restrict__ perm_old, const uint32_t* __restrict__ pos_old,
    int32_t* __restrict__ perm_new, uint32_t* __restrict__ pos_new) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int bg = blockIdx.y;
    if (p >= D.rcap) return;
    const int b = bg / D.Hkv;
    const int old_nr = lo.v[b] - D.n_sink, new_nr = hi.v[b] - D.n_sink;
    const int64_t row = static_cast<int64_t>(bg) * D.rcap;
    if (p < old_nr) {
        const uint32_t w = pos_old[row + p];
        const int q = p + shift[static_cast<int64_t>(bg) * D.n_list + static_cast<int>(w >> kPosBits)];
        perm_new[row + q] = perm_old[row + p];
        pos_new[row + q] = w;
    } else if (p >= new_nr) {
        perm_new[row + p] = -1;
        pos_new[row + p] = 0u;
    }
}

// check_ids_kernel: the smallest flat index (b, g, token) of R whose list id
// lies outside [0, n_list), by atomicMin into `bad` (left at all ones when
// every id is valid).
__global__ __launch_bounds__(256) void check_ids_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                        const int32_t* __restrict__ ids_tm,
                                                        unsigned long long* bad) {
    const int bg = blockIdx.y;
    const int b = bg / D.Hkv;
    const int t = lo.v[b] + blockIdx.x * 256 + threadIdx.x;
    if (t >= hi.v[b]) return;
    const int64_t at = static_cast<int64_t>(bg) * D.rcap + t;
    const int32_t j = ids_tm[at];
    if (j < 0 || j >= D.n_list) atomicMin(bad, static_cast<unsigned long long>(at));
}

// finish_lists_kernel: after the grouping of R_b by list (perm, loff), the
// list word of every position and the cleared positions past |R_b|.
__global__ __launch_bounds__(256) void finish_lists_kernel(Dims D, BatchInts lo, BatchInts hi,
                                                           const int32_t* __restrict__ ids_tm,
                                                           int32_t* __restrict__ perm,
                                                           uint32_t* __restrict__ pos_word,
                                                           int32_t* __restrict__ n_r_dev,
                                                           int32_t* __restrict__ n_seq_dev) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int bg = blockIdx.y;
    const int b = bg / D.Hkv;
    if (p == 0 && bg % D.Hkv == 0) {
        n_r_dev[b] = hi.v[b] - D.n_sink;
        n_seq_dev[b] = hi.v[b] + D.n_local;
    }
    if (p >= D.rcap) return;
    const int64_t row = static_cast<int64_t>(bg) * D.rcap;
    if (p < hi.v[b] - lo.v[b]) {
        const int t = perm[row + p];
        const int j = min(max(ids_tm[row + t], 0), D.n_list - 1);
        pos_word[row + p] = (static_cast<uint32_t>(j) << kPosBits) | static_cast<uint32_t>(t);
    } else {
        perm[row + p] = -1;
        pos_word[row + p] = 0u;
    }
}

hipError_t launch_sort_lists(const Dims& D, const BatchInts& lo, const BatchInts& hi, int max_n,
                             const int32_t* ids_tm, const int32_t* zero_loff, int32_t* loff,
                             int32_t* shift, int32_t* perm, uint32_t* pos_word,
                             int32_t* n_r_dev, int32_t* n_seq_dev, unsigned long long* bad,
                             int32_t* scratch, size_t scratch_ints, hipStream_t s) {
    if (max_n > 0) {
        hipLaunchKernelGGL(check_ids_kernel, dim3((max_n + 255) / 256, D.B * D.Hkv), dim3(256), 0, s,
                           D, lo, hi, ids_tm, bad);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const size_t nseg = (static_cast<size_t>(max_n) + kBuildSegTok - 1) / kBuildSegTok;
    if (D.n_list <= 1024 && scratch &&
        nseg * static_cast<size_t>(D.B) * D.Hkv * D.n_list <= scratch_ints) {
        // the build's segmented grouping, many workgroups per (b, g)
        hipError_t e = launch_group_segments(D, lo, hi, 0, ids_tm, nullptr, scratch, perm, loff, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(finish_lists_kernel, dim3((D.rcap + 255) / 256, D.B * D.Hkv), dim3(256), 0, s,
                           D, lo, hi, ids_tm, perm, pos_word, n_r_dev, n_seq_dev);
        return hipGetLastError();
    }
    // a merge into an empty index: every token of R is new (old offsets all
    // zero, no old positions to move)
    hipLaunchKernelGGL(update_lists_kernel, dim3(D.B * D.Hkv), dim3(kListThreads), 0, s, D, lo, hi,
                       ids_tm, zero_loff, loff, shift, perm, pos_word, n_r_dev, n_seq_dev);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // positions past |R_b| are cleared
    hipLaunchKernelGGL(shift_positions_kernel, dim3((D.rcap + 255) / 256, D.B * D.Hkv), dim3(256), 0,
                       s, D, lo, hi, shift, nullptr, nullptr, perm, pos_word);
    return hipGetLastError();
}

hipError_t launch_update_lists(const Dims& D, const BatchInts& lo, const BatchInts& hi,
                               const KV& kv, const int32_t* ids_tm, const int32_t* old_loff,
                               const int32_t* perm_old, const uint32_t* pos_old, int32_t* new_loff,
                               int32_t* shift, int32_t* perm_new, uint32_t* pos_new,
                               int32_t* n_r_dev, int32_t* n_seq_dev,
                               float* means, double* sums, hipStream_t s) {
    hipLaunchKernelGGL(update_lists_kernel, dim3(D.B * D.Hkv), dim3(kListThreads), 0, s, D, lo, hi,
                       ids_tm, old_loff, new_loff, shift, perm_new, pos_new, n_r_dev, n_seq_dev);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(shift_positions_kernel, dim3((D.rcap + 255) / 256, D.B * D.Hkv), dim3(256), 0,
                       s, D, lo, hi, shift, perm_old, pos_old, perm_new, pos_new);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid(D.n_list, D.Hkv, D.B);
    if (kv.bf16)
        hipLaunchKernelGGL(means_update_kernel<bf16_t>, grid, dim3(kHeadDim), 0, s, D,
                           static_cast<const bf16_t*>(kv.v), kv.sb, kv.sh, kv.sn, old_loff, new_loff,
                           perm_new, means, sums);
    else
        hipLaunchKernelGGL(means_update_kernel<float>, grid, dim3(kHeadDim), 0, s, D,
                           static_cast<const float*>(kv.v), kv.sb, kv.sh, kv.sn, old_loff, new_loff,
                           perm_new, means, sums);
    return hipGetLastError();
}

hipError_t launch_encode_update(const Dims& D, const BatchInts& lo, const BatchInts& hi,
                                int max_new, const KV& kv, const float* centroids,
                                const float* codebooks, int32_t* ids_tm, uint8_t* codes_tm,
                                float* norms_tm, hipStream_t s) {
    if (max_new <= 0) return hipSuccess;
    const dim3 grid(max_new, D.Hkv, D.B);
#define PQHSA_ENC1(TT, PQT)                                                                     \
    hipLaunchKernelGGL((encode_one_kernel<TT, PQT>), grid, dim3(kEncThreads), 0, s, D, lo, hi,    \
                       static_cast<const TT*>(kv.k), kv.sb, kv.sh, kv.sn, centroids, codebooks,   \
                       ids_tm, codes_tm, norms_tm)
    if (kv.bf16) {
        if (D.pq_bits == 4) PQHSA_ENC1(bf16_t, Pq4); else PQHSA_ENC1(bf16_t, Pq8);
    } else {
        if (D.pq_bits == 4) PQHSA_ENC1(float, Pq4); else PQHSA_ENC1(float, Pq8);
    }
#undef PQHSA_ENC1
    return hipGetLastError();
}

}  // namespace pqhsa
