// Exact attention over E = S u L u T, the per-list background, and the final
// merge (Section 3.2, Eqs. 4-5), plus the dense decode baseline.
//
// Every partial result is a triple (m, Z, N[d]) meaning "sum of
// exp(logit - m) = Z, sum of exp(logit - m) v = N"; partials combine by the
// usual log-sum-exp rule, so the common shift m0 of Section 3.2 never has to
// be known in advance.
//
//  * attend_kernel, exact role: one workgroup per (row, split of kAttnRows
//    rows of E). 16 lanes hold one K/V row (8 elements each); a wave keeps 4
//    rows in flight and runs an online softmax per 16-lane group.
//  * attend_kernel, background role: one workgroup per (batch element, KV
//    head, kBgLists lists). For each list j and each of the G query heads:
//    M_j = (below-threshold mass of the scan segments) * exp(tau_lo - shift)
//          + (unselected-candidate mass of the top-k stage),
//    then Z_B += M_j and N_B += M_j * v_bar_j (Eq. 4), reading each list mean
//    once for the whole group.
//  * merge_kernel: log-sum-exp of all partials of a row, y = N / Z (Eq. 5).
#include "device_common.h"
#include "pqhsa_internal.h"

namespace pqhsa {

constexpr int kAttnThreads = 256;    // 4 waves x 4 groups of 16 lanes = 16 row streams
constexpr int kStreams = kAttnThreads / 16;

struct Online {
    float m, z, acc[8];
};

__device__ __forceinline__ void online_init(Online& o) {
    o.m = -__builtin_huge_valf();
    o.z = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) o.acc[t] = 0.0f;
}

__device__ __forceinline__ void online_push(Online& o, float logit, const float (&v)[8]) {
    const float m_new = fmaxf(o.m, logit);
    const float a = __expf(o.m - m_new);   // 0 when o.m = -inf
    const float p = __expf(logit - m_new);
    o.z = o.z * a + p;
#pragma unroll
    for (int t = 0; t < 8; ++t) o.acc[t] = o.acc[t] * a + p * v[t];
    o.m = m_new;
}

// Combine the 16 streams of a workgroup into one partial written at `dst`.
// Must be called by all threads.
__device__ __forceinline__ void block_combine(const Online& o, float* sm, float* sz, float* sacc,
                                              float* __restrict__ dst) {
    const int stream = threadIdx.x >> 4;
    const int lane16 = threadIdx.x & 15;
    if (lane16 == 0) {
        sm[stream] = o.m;
        sz[stream] = o.z;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) sacc[stream * kHeadDim + lane16 * 8 + t] = o.acc[t];
    __syncthreads();
    if (threadIdx.x < kHeadDim) {
        const int t = threadIdx.x;
        float M = -__builtin_huge_valf();
        for (int s = 0; s < kStreams; ++s) M = fmaxf(M, sm[s]);
        float Z = 0.0f, N = 0.0f;
        if (M != -__builtin_huge_valf()) {
            for (int s = 0; s < kStreams; ++s) {
                const float f = __expf(sm[s] - M);
                Z += sz[s] * f;
                N += sacc[s * kHeadDim + t] * f;
            }
        }
        if (t == 0) {
            dst[0] = M;
            dst[1] = Z;
        }
        dst[4 + t] = N;
    }
    __syncthreads();
}

template <typename T, int G>
__global__ __launch_bounds__(kAttnThreads) void attend_kernel(Dims D, BatchInts tk, KV kv,
                                                              Index ix, Work w, int nsplit_max,
                                                              int n_bgc) {
    __shared__ float sm[kStreams], sz[kStreams];
    // [16 streams][d] for the exact role, [4 waves][G][d] for the background role
    __shared__ float sacc[(kStreams > 4 * G ? kStreams : 4 * G) * kHeadDim];
    const int n_exact_wg = D.B * D.Hq * nsplit_max;
    const int P = nsplit_max + n_bgc;
    const int lane16 = threadIdx.x & 15;
    const int stream = threadIdx.x >> 4;

    if (static_cast<int>(blockIdx.x) < n_exact_wg) {
        // ---------------- exact attention over a split of E ----------------
        const int row = blockIdx.x / nsplit_max;
        const int split = blockIdx.x % nsplit_max;
        const int b = row / D.Hq;
        const int h = row % D.Hq;
        const int g = h / G;
        const int k = tk.v[b];
        const int n_seq = ix.n_seq[b];
        const int nE = D.n_sink + D.n_local + k;
        const int e0 = split * kAttnRows;
        if (e0 >= nE) return;   // the merge reads only the splits that exist
        const int e1 = min(e0 + kAttnRows, nE);
        const T* qp = static_cast<const T*>(kv.q) + static_cast<int64_t>(row) * kHeadDim + lane16 * 8;
        float qv[8];
        Load8<T>::run(qp, qv);
        const T* kb = static_cast<const T*>(kv.k) + b * kv.sb + g * kv.sh + lane16 * 8;
        const T* vb = static_cast<const T*>(kv.v) + b * kv.sb + g * kv.sh + lane16 * 8;
        const int32_t* sel = w.sel_tok + static_cast<int64_t>(row) * D.max_topk;
        const int local0 = n_seq - D.n_local;
        Online o;
        online_init(o);
        for (int e = e0 + stream; e < e1; e += kStreams) {
            int tok;
            if (e < D.n_sink) tok = e;
            else if (e < D.n_sink + D.n_local) tok = local0 + (e - D.n_sink);
            else tok = sel[e - D.n_sink - D.n_local];
            tok = min(max(tok, 0), n_seq - 1);   // never read outside the sequence
            float kf[8], vf[8];
            Load8<T>::run(kb + tok * kv.sn, kf);
            Load8<T>::run(vb + tok * kv.sn, vf);
            float dot = 0.0f;
#pragma unroll
            for (int t = 0; t < 8; ++t) dot = fmaf(qv[t], kf[t], dot);
            dot = sum16(dot);
            online_push(o, dot * D.inv_sqrt_d, vf);
        }
        block_combine(o, sm, sz, sacc,
                      w.partial + (static_cast<int64_t>(row) * P + split) * kPartStride);
        return;
    }

    // ---------------- per-list background (Eq. 4) ----------------
    __shared__ float bz[4][G];
    const int idx = blockIdx.x - n_exact_wg;
    const int bg = idx / n_bgc;
    const int lc = idx % n_bgc;
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;
    const int row0 = b * D.Hq + g * G;
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const float neg_inf = -__builtin_huge_valf();

    float shift[G], below_scale[G];
    bool live[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        shift[hh] = w.row_shift[row0 + hh];
        const float tlo = w.tau_lo[row0 + hh];
        live[hh] = shift[hh] != neg_inf;
        const bool use_below = live[hh] && tlo != neg_inf && w.row_flag[row0 + hh] == 0;
        below_scale[hh] = use_below ? __expf(tlo - shift[hh]) : 0.0f;
    }
    float Z[G], N[G][2];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) { Z[hh] = 0.0f; N[hh][0] = 0.0f; N[hh][1] = 0.0f; }

    const int j0 = lc * kBgLists;
    const int j1 = min(j0 + kBgLists, D.n_list);
    const int32_t* seg0 = ix.seg0 + static_cast<int64_t>(bg) * (D.n_list + 1);
    const float* segs = w.seg_sum + static_cast<int64_t>(bg) * D.nseg_cap * G;
    for (int j = j0 + wave; j < j1; j += kAttnThreads / kWave) {
        const int s0 = seg0[j], s1 = seg0[j + 1];
        const float2 vbar = *reinterpret_cast<const float2*>(
            ix.means + (static_cast<int64_t>(bg) * D.n_list + j) * kHeadDim + 2 * lane);
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float below = 0.0f;
            for (int s = s0; s < s1; ++s) below += segs[s * G + hh];
            float Mj = below * below_scale[hh] +
                       w.cand_mass[static_cast<int64_t>(row0 + hh) * D.n_list + j];
            if (!live[hh]) Mj = 0.0f;
            Z[hh] += Mj;
            N[hh][0] = fmaf(Mj, vbar.x, N[hh][0]);
            N[hh][1] = fmaf(Mj, vbar.y, N[hh][1]);
        }
    }
    // combine the 4 waves (sacc reused as [4][G][128])
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        sacc[(wave * G + hh) * kHeadDim + 2 * lane] = N[hh][0];
        sacc[(wave * G + hh) * kHeadDim + 2 * lane + 1] = N[hh][1];
        if (lane == 0) bz[wave][hh] = Z[hh];
    }
    __syncthreads();
    if (threadIdx.x < kHeadDim) {
        const int t = threadIdx.x;
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float n = 0.0f, z = 0.0f;
#pragma unroll
            for (int wv = 0; wv < 4; ++wv) {
                n += sacc[(wv * G + hh) * kHeadDim + t];
                z += bz[wv][hh];
            }
            float* dst = w.partial + (static_cast<int64_t>(row0 + hh) * P + nsplit_max + lc) * kPartStride;
            if (t == 0) {
                dst[0] = shift[hh];
                dst[1] = z;
            }
            dst[4 + t] = n;
        }
    }
}

// y = (sum of partials' N) / (sum of partials' Z) under one shift (Eq. 5).
__global__ __launch_bounds__(kHeadDim) void merge_kernel(Dims D, BatchInts n_exact_parts,
                                                         const float* __restrict__ partial,
                                                         int P, int first_bg, int n_bg,
                                                         float* __restrict__ out) {
    const int row = blockIdx.x;
    const int b = row / D.Hq;
    const int t = threadIdx.x;
    const float* pr = partial + static_cast<int64_t>(row) * P * kPartStride;
    const int ne = n_exact_parts.v[b];
    float M = -__builtin_huge_valf();
    for (int p = 0; p < ne; ++p) M = fmaxf(M, pr[p * kPartStride]);
    for (int p = 0; p < n_bg; ++p) {
        const float* q = pr + (first_bg + p) * kPartStride;
        if (q[1] > 0.0f) M = fmaxf(M, q[0]);
    }
    float Z = 0.0f, N = 0.0f;
    for (int p = 0; p < ne; ++p) {
        const float* q = pr + p * kPartStride;
        const float f = __expf(q[0] - M);
        Z += q[1] * f;
        N += q[4 + t] * f;
    }
    for (int p = 0; p < n_bg; ++p) {
        const float* q = pr + (first_bg + p) * kPartStride;
        if (q[1] > 0.0f) {
            const float f = __expf(q[0] - M);
            Z += q[1] * f;
            N += q[4 + t] * f;
        }
    }
    out[static_cast<int64_t>(row) * kHeadDim + t] = N / Z;
}

template <typename T, int G>
static hipError_t launch_attend_t(const Dims& D, const BatchInts& tk, const KV& kv,
                                  const Index& ix, const Work& w, int nsplit_max, hipStream_t s) {
    const int n_bgc = (D.n_list + kBgLists - 1) / kBgLists;
    const int grid = D.B * D.Hq * nsplit_max + D.B * D.Hkv * n_bgc;
    hipLaunchKernelGGL((attend_kernel<T, G>), dim3(grid), dim3(kAttnThreads), 0, s, D, tk, kv,
                       ix, w, nsplit_max, n_bgc);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_attend_g(const Dims& D, const BatchInts& tk, const KV& kv,
                                  const Index& ix, const Work& w, int nsplit_max, hipStream_t s) {
    switch (D.G) {
        case 1: return launch_attend_t<T, 1>(D, tk, kv, ix, w, nsplit_max, s);
        case 2: return launch_attend_t<T, 2>(D, tk, kv, ix, w, nsplit_max, s);
        case 4: return launch_attend_t<T, 4>(D, tk, kv, ix, w, nsplit_max, s);
        case 8: return launch_attend_t<T, 8>(D, tk, kv, ix, w, nsplit_max, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attend(const Dims& D, const BatchInts& tk, const KV& kv, const Index& ix,
                         const Work& w, int nsplit_max, hipStream_t s) {
    return kv.bf16 ? launch_attend_g<bf16_t>(D, tk, kv, ix, w, nsplit_max, s)
                   : launch_attend_g<float>(D, tk, kv, ix, w, nsplit_max, s);
}

hipError_t launch_merge(const Dims& D, const BatchInts& tk, const Work& w, float* out,
                        int nsplit_max, hipStream_t s) {
    BatchInts ne;
    for (int b = 0; b < D.B; ++b) {
        const int nE = D.n_sink + D.n_local + tk.v[b];
        ne.v[b] = (nE + kAttnRows - 1) / kAttnRows;
    }
    const int n_bgc = (D.n_list + kBgLists - 1) / kBgLists;
    hipLaunchKernelGGL(merge_kernel, dim3(D.B * D.Hq), dim3(kHeadDim), 0, s, D, ne, w.partial,
                       nsplit_max + n_bgc, nsplit_max, n_bgc, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Dense decode baseline: every cached row, all G heads of a group per K/V load.
// ---------------------------------------------------------------------------
template <typename T, int G>
__global__ __launch_bounds__(kAttnThreads) void dense_kernel(Dims D, KV kv, BatchInts lens,
                                                             float* __restrict__ partial,
                                                             int nsplit_max) {
    __shared__ float sm[kStreams], sz[kStreams];
    __shared__ float sacc[kStreams * kHeadDim];
    const int bg = blockIdx.x / nsplit_max;
    const int split = blockIdx.x % nsplit_max;
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;
    const int n = lens.v[b];
    const int t0 = split * kDenseRows;
    if (t0 >= n) return;
    const int t1 = min(t0 + kDenseRows, n);
    const int lane16 = threadIdx.x & 15;
    const int stream = threadIdx.x >> 4;
    float qv[G][8];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
        Load8<T>::run(static_cast<const T*>(kv.q) +
                          (static_cast<int64_t>(b) * D.Hq + g * G + hh) * kHeadDim + lane16 * 8,
                      qv[hh]);
    const T* kb = static_cast<const T*>(kv.k) + b * kv.sb + g * kv.sh + lane16 * 8;
    const T* vb = static_cast<const T*>(kv.v) + b * kv.sb + g * kv.sh + lane16 * 8;
    Online o[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) online_init(o[hh]);
    for (int t = t0 + stream; t < t1; t += kStreams) {
        float kf[8], vf[8];
        Load8<T>::run(kb + t * kv.sn, kf);
        Load8<T>::run(vb + t * kv.sn, vf);
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float dot = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) dot = fmaf(qv[hh][i], kf[i], dot);
            dot = sum16(dot);
            online_push(o[hh], dot * D.inv_sqrt_d, vf);
        }
    }
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
        block_combine(o[hh], sm, sz, sacc,
                      partial + ((static_cast<int64_t>(b) * D.Hq + g * G + hh) * nsplit_max + split) *
                                    kPartStride);
}

template <typename T, int G>
static hipError_t launch_dense_t(const Dims& D, const KV& kv, const BatchInts& lens,
                                 float* partial, int nsplit_max, hipStream_t s) {
    hipLaunchKernelGGL((dense_kernel<T, G>), dim3(D.B * D.Hkv * nsplit_max), dim3(kAttnThreads), 0,
                       s, D, kv, lens, partial, nsplit_max);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_dense_g(const Dims& D, const KV& kv, const BatchInts& lens,
                                 float* partial, int nsplit_max, hipStream_t s) {
    switch (D.G) {
        case 1: return launch_dense_t<T, 1>(D, kv, lens, partial, nsplit_max, s);
        case 2: return launch_dense_t<T, 2>(D, kv, lens, partial, nsplit_max, s);
        case 4: return launch_dense_t<T, 4>(D, kv, lens, partial, nsplit_max, s);
        case 8: return launch_dense_t<T, 8>(D, kv, lens, partial, nsplit_max, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_dense(const Dims& D, const KV& kv, const BatchInts& lens, float* partial,
                        float* out, int nsplit_max, hipStream_t s) {
    hipError_t e = kv.bf16 ? launch_dense_g<bf16_t>(D, kv, lens, partial, nsplit_max, s)
                           : launch_dense_g<float>(D, kv, lens, partial, nsplit_max, s);
    if (e != hipSuccess) return e;
    BatchInts ne;
    for (int b = 0; b < D.B; ++b) ne.v[b] = (lens.v[b] + kDenseRows - 1) / kDenseRows;
    hipLaunchKernelGGL(merge_kernel, dim3(D.B * D.Hq), dim3(kHeadDim), 0, s, D, ne, partial,
                       nsplit_max, 0, 0, out);
    return hipGetLastError();
}

}  // namespace pqhsa
