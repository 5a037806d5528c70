// LUT build (Section 3.1, Eq. 2): per (batch element, KV head) the fine table
// F[m][z][hh] = (q_hh^(m) . p_{m,z}) / sqrt(d) for the G query heads of the
// group, and the coarse table C[j][hh] = (q_hh . c_j) / sqrt(d).
//
// Folding r_q / sqrt(d) into the tables: (r_q / sqrt(d)) u_q . x = q . x / sqrt(d),
// so the tables are built from q / sqrt(d) directly and no normalisation of q
// is needed (a zero query gives all-zero tables, hence zero scores).
#include "device_common.h"
#include "pqhsa_internal.h"

namespace pqhsa {

constexpr int kLutThreads = 256;
constexpr int kCoarseLists = 64;   // lists per coarse workgroup

template <typename T, int G>
__global__ __launch_bounds__(kLutThreads) void lut_kernel(Dims D, const T* __restrict__ q,
                                                          const float* __restrict__ codebooks,
                                                          const float* __restrict__ centroids,
                                                          float* __restrict__ lut,
                                                          float* __restrict__ coarse) {
    const int n_coarse = (D.n_list + kCoarseLists - 1) / kCoarseLists;
    const int per_bg = kPqM + n_coarse;
    const int bg = blockIdx.x / per_bg;
    const int part = blockIdx.x % per_bg;
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;
    const T* qg = q + (static_cast<int64_t>(b) * D.Hq + g * G) * kHeadDim;

    if (part < kPqM) {
        // fine table of subspace m: one codeword per thread
        const int m = part;
        const int z = threadIdx.x;
        float qs[G][kDsub];
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
#pragma unroll
            for (int t = 0; t < kDsub; ++t)
                qs[hh][t] = load1(qg + hh * kHeadDim + m * kDsub + t) * D.inv_sqrt_d;
        const float* p = codebooks + ((static_cast<int64_t>(bg) * kPqM + m) * kKsub + z) * kDsub;
        const float4 p0 = *reinterpret_cast<const float4*>(p);
        const float4 p1 = *reinterpret_cast<const float4*>(p + 4);
        const float pv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
        float* o = lut + ((static_cast<int64_t>(bg) * kPqM + m) * kKsub + z) * G;
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float acc = 0.0f;
#pragma unroll
            for (int t = 0; t < kDsub; ++t) acc = fmaf(qs[hh][t], pv[t], acc);
            o[hh] = acc;
        }
        return;
    }

    // coarse table: 16 lanes per list, 8 dimensions per lane
    const int c = part - kPqM;
    const int lane16 = threadIdx.x & 15;
    const int group = threadIdx.x >> 4;   // 16 groups of 16 lanes
    float qc[G][8];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
        for (int t = 0; t < 8; ++t)
            qc[hh][t] = load1(qg + hh * kHeadDim + lane16 * 8 + t) * D.inv_sqrt_d;
    // all centroid slices of this thread first, then the dot products
    constexpr int kPer = kCoarseLists / (kLutThreads / 16);
    float4 cv[kPer][2];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int j = c * kCoarseLists + group + u * (kLutThreads / 16);
        const int jc = j < D.n_list ? j : D.n_list - 1;   // keep all lanes active
        const float* cp = centroids + (static_cast<int64_t>(bg) * D.n_list + jc) * kHeadDim + lane16 * 8;
        cv[u][0] = *reinterpret_cast<const float4*>(cp);
        cv[u][1] = *reinterpret_cast<const float4*>(cp + 4);
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int j = c * kCoarseLists + group + u * (kLutThreads / 16);
        const float cf[8] = {cv[u][0].x, cv[u][0].y, cv[u][0].z, cv[u][0].w,
                             cv[u][1].x, cv[u][1].y, cv[u][1].z, cv[u][1].w};
        float mine = 0.0f;
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float acc = 0.0f;
#pragma unroll
            for (int t = 0; t < 8; ++t) acc = fmaf(qc[hh][t], cf[t], acc);
            acc = sum16(acc);
            if (lane16 == hh) mine = acc;
        }
        if (j < D.n_list && lane16 < G)
            coarse[(static_cast<int64_t>(bg) * D.n_list + j) * G + lane16] = mine;
    }
}

template <typename T, int G>
static hipError_t launch_lut_t(const Dims& D, const KV& kv, const Index& ix, const Work& w,
                               hipStream_t s) {
    const int n_coarse = (D.n_list + kCoarseLists - 1) / kCoarseLists;
    const int grid = D.B * D.Hkv * (kPqM + n_coarse);
    hipLaunchKernelGGL((lut_kernel<T, G>), dim3(grid), dim3(kLutThreads), 0, s, D,
                       static_cast<const T*>(kv.q), ix.codebooks, ix.centroids, w.lut,
                       w.coarse);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_lut_g(const Dims& D, const KV& kv, const Index& ix, const Work& w,
                               hipStream_t s) {
    switch (D.G) {
        case 1: return launch_lut_t<T, 1>(D, kv, ix, w, s);
        case 2: return launch_lut_t<T, 2>(D, kv, ix, w, s);
        case 4: return launch_lut_t<T, 4>(D, kv, ix, w, s);
        case 8: return launch_lut_t<T, 8>(D, kv, ix, w, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_lut(const Dims& D, const KV& kv, const Index& ix, const Work& w,
                      hipStream_t s) {
    return kv.bf16 ? launch_lut_g<bf16_t>(D, kv, ix, w, s) : launch_lut_g<float>(D, kv, ix, w, s);
}

}  // namespace pqhsa
