// Decode prologue: the LUT build (Section 3.1, Eq. 2) and the candidate
// threshold sample, in one launch with two workgroup roles.
//
// LUT role, per (batch element, KV head) and part: the fine table
// F[m][z][hh] = (q_hh^(m) . p_{m,z}) / sqrt(d) for the G query heads of the
// group (read by the scan, the next launch; also written head-major for the
// sample role), and the coarse table C[j][hh] = (q_hh . c_j) / sqrt(d).
// Folding r_q / sqrt(d) into the tables: (r_q / sqrt(d)) u_q . x = q . x / sqrt(d),
// so the tables are built from q / sqrt(d) directly and no normalisation of q
// is needed (a zero query gives all-zero tables, hence zero scores).
// Each LUT workgroup writes what the sample role reads with device-scope
// stores and, once they are acknowledged, sets its own flag to the call's
// epoch (read at kernel start from a device counter that the call's last
// kernel advances).
//
// Sample role, per (batch element, query head) row: scores a stratified
// sample of the row's list-major positions (contiguous runs of kSampleRun
// positions, evenly spread) and takes a sample order statistic as the
// candidate threshold tau_lo, chosen so that about twice k tokens of the
// whole row score at or above it. The role issues its sample loads, then
// waits for its KV head's LUT parts (every LUT workgroup has a lower
// workgroup id and waits for nothing, so it is dispatched first and
// finishes), then reads its head's fine table and the coarse terms of its
// samples.
//
// When a call's budgets and lengths are device data, the sample role reads
// them from the caller's arrays, clamps them, and the first query head of
// each sequence writes them to the workspace for the later kernels.
//
// Any threshold gives the same final output: it only decides how many
// candidates the scan emits (the top-k stage falls back to an exact re-scan
// when fewer than k tokens reach it). So the wait is bounded: a sample
// workgroup that does not see its tables within kSpinLimit polls sets
// tau_lo = -inf, which makes every token a candidate, and exits.
#include <type_traits>

#include "device_common.h"
#include "hist_select.h"
#include "pq_score.h"
#include "pqhsa_internal.h"
#include "radix_select.h"

namespace pqhsa {

constexpr int kProThreads = 512;
constexpr int kFineWg = kProThreads / Pq8::K;              // Pq8 subspaces per fine workgroup: 2
constexpr int kCoarseGroups = kProThreads / 16;            // 16-lane groups
constexpr int kCoarsePer = kCoarseLists / kCoarseGroups;   // lists per group: 2
constexpr int kSamplesPer = kMaxSamples / kProThreads;     // samples per thread: 4
constexpr int kPolls = 2;                                  // counter reads in flight
constexpr int kPollSleep = 8;                              // between reads: 8 x 64 clocks
constexpr int kFlagsPerLane = 3;                           // LUT part flags per lane of the poll
static_assert(8 + kMaxLists / kCoarseLists <= kFlagsPerLane * kWave, "LUT parts per KV head");
constexpr int kSpinLimit = 1 << 16;                        // poll rounds before giving up
static_assert(kFineWg * Pq8::K == kProThreads && Pq8::M / kFineWg == 8, "Pq8 fine tiling");
static_assert(Pq4::LUT_ROW <= kProThreads, "Pq4 fine table: one codeword per thread");
static_assert(kCoarsePer * kCoarseGroups == kCoarseLists, "coarse tiling");
static_assert(kSamplesPer * kProThreads == kMaxSamples && kMaxSamples % kSampleRun == 0, "samples");

// (q / sqrt(d)) . c over 16 lanes of 8 dimensions each; every lane of the
// 16-lane group receives the same sum.
__device__ __forceinline__ float coarse_entry(const float (&qc)[8], const float4 c0,
                                             const float4 c1) {
    const float cf[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc = fmaf(qc[t], cf[t], acc);
    return sum16(acc);
}

// One fine-table entry (q^(m) / sqrt(d)) . p_{m,z} over the DSUB dimensions of
// subspace m (qm points at them).
template <typename T, int DSUB>
__device__ __forceinline__ float fine_entry(const T* qm, const float (&pv)[DSUB], float inv_sqrt_d) {
    float acc = 0.0f;
#pragma unroll
    for (int t0 = 0; t0 < DSUB; t0 += 8) {
        float qs[8];
        Load8<T>::run(qm + t0, qs);
#pragma unroll
        for (int t = 0; t < 8; ++t) acc = fmaf(qs[t] * inv_sqrt_d, pv[t0 + t], acc);
    }
    return acc;
}

template <int DSUB>
__device__ __forceinline__ void load_codeword(const float* p, float (&pv)[DSUB]) {
#pragma unroll
    for (int t = 0; t < DSUB; t += 4) {
        const float4 v = *reinterpret_cast<const float4*>(p + t);
        pv[t] = v.x; pv[t + 1] = v.y; pv[t + 2] = v.z; pv[t + 3] = v.w;
    }
}

// Store G consecutive floats.
template <int G>
__device__ __forceinline__ void store_g(float* o, const float (&e)[G]) {
    if constexpr (G == 8) {
        reinterpret_cast<float4*>(o)[0] = make_float4(e[0], e[1], e[2], e[3]);
        reinterpret_cast<float4*>(o)[1] = make_float4(e[4], e[5], e[6], e[7]);
    } else if constexpr (G == 4) {
        *reinterpret_cast<float4*>(o) = make_float4(e[0], e[1], e[2], e[3]);
    } else if constexpr (G == 2) {
        *reinterpret_cast<float2*>(o) = make_float2(e[0], e[1]);
    } else {
        o[0] = e[0];
    }
}

template <typename T, int G, typename PQ>
__device__ __forceinline__ void lut_role(const Dims& D, const T* __restrict__ q,
                                         const float* __restrict__ codebooks,
                                         const float* __restrict__ centroids, const Work& w,
                                         int bg, int part) {
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;
    const int row0 = b * D.Hq + g * G;
    const T* qg = q + static_cast<int64_t>(row0) * kHeadDim;
    const int tid = threadIdx.x;
    // this call's epoch for the KV head (see sample_role), needed at the end
    const uint32_t ep = tid == 0 ? counter_read(w.epoch + bg) + 1u : 0u;
    const int fine_parts = prologue_fine_parts(PQ::BITS);
    if (part < fine_parts) {
        // fine table: one (subspace, codeword) per thread (Pq8: 2 subspaces
        // per part; Pq4: the whole table, 128 codewords, in one part)
        const int e_id = std::is_same<PQ, Pq8>::value ? part * kProThreads + tid : tid;
        if (e_id < PQ::LUT_ROW) {
            const int m = e_id / PQ::K;
            const int z = e_id % PQ::K;
            float pv[PQ::DSUB];
            load_codeword<PQ::DSUB>(codebooks + (static_cast<int64_t>(bg) * PQ::LUT_ROW + e_id) * PQ::DSUB, pv);
            float* o = w.lut + (static_cast<int64_t>(bg) * PQ::LUT_ROW + e_id) * G;
            float e[G];
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                e[hh] = fine_entry<T, PQ::DSUB>(qg + hh * kHeadDim + m * PQ::DSUB, pv, D.inv_sqrt_d);
                store_device(w.lut_head + static_cast<int64_t>(row0 + hh) * PQ::LUT_ROW + m * PQ::K + z,
                             e[hh]);
            }
            store_g<G>(o, e);   // read by the next launch only: plain stores
        }
    } else {
        // coarse table: 16 lanes per list, 8 dimensions per lane
        const int c = part - fine_parts;
        const int lane16 = tid & 15;
        const int group = tid >> 4;
        float4 cv[kCoarsePer][2];
#pragma unroll
        for (int u = 0; u < kCoarsePer; ++u) {
            const int j = c * kCoarseLists + group + u * kCoarseGroups;
            const int jc = j < D.n_list ? j : D.n_list - 1;   // keep all lanes active
            const float* cp = centroids + (static_cast<int64_t>(bg) * D.n_list + jc) * kHeadDim + lane16 * 8;
            cv[u][0] = *reinterpret_cast<const float4*>(cp);
            cv[u][1] = *reinterpret_cast<const float4*>(cp + 4);
        }
        float qc[G][8];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            Load8<T>::run(qg + hh * kHeadDim + lane16 * 8, qc[hh]);
#pragma unroll
            for (int t = 0; t < 8; ++t) qc[hh][t] *= D.inv_sqrt_d;
        }
#pragma unroll
        for (int u = 0; u < kCoarsePer; ++u) {
            const int j = c * kCoarseLists + group + u * kCoarseGroups;
            float mine = 0.0f;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                const float acc = coarse_entry(qc[hh], cv[u][0], cv[u][1]);
                if (lane16 == hh) mine = acc;
            }
            if (j < D.n_list && lane16 < G)
                store_device(w.coarse + (static_cast<int64_t>(bg) * D.n_list + j) * G + lane16, mine);
        }
    }
    // publish: every store acknowledged at device scope, then this part's
    // flag takes the call's epoch (a plain device-scope store: the parts of a
    // KV head never contend on one address)
    wait_vector_memory();
    __syncthreads();
    if (tid == 0) store_device(w.lut_flag + bg * prologue_parts(D.n_list, PQ::BITS) + part, ep);
}

struct SampleLds {
    float lut[kLutRowMax];   // the head's fine table [M][K]
    int hist[kHistBins];
    int ready;
    SelectScratch ss;
    BlockScratch bs;
};

template <typename T, int G, typename PQ, bool kDev>
__device__ __forceinline__ void sample_role(const Dims& D, const BatchArgs& ba, const Index& ix,
                                            const Work& w, float bias, int row,
                                            SampleLds& sm) {
    const int tid = threadIdx.x;
    const int b = row / D.Hq;
    const int h = row % D.Hq;
    const int g = h / G;
    const int hh = h % G;
    const int bg = b * D.Hkv + g;
    int n_r, k;
    if constexpr (kDev) {
        // the call's integers from the caller's device arrays, published for
        // the later kernels by the first query head of each sequence
        const SeqArgs a = clamp_seq_args(D, ix.n_r[b], w.dev_lens[b], w.dev_topk[b]);
        n_r = a.n_r;
        k = a.topk;
        if (h == 0 && tid == 0) {
            w.ba_dev->topk[b] = a.topk;
            w.ba_dev->n_r[b] = a.n_r;
            w.ba_dev->n_tail[b] = a.n_tail;
        }
    } else {
        n_r = ba.n_r[b];
        k = ba.topk[b];
    }
    const float neg_inf = -__builtin_huge_valf();
    if (n_r == 0) {
        if (tid == 0) {
            w.tau_lo[row] = neg_inf;
            w.tau_hi[row] = neg_inf;
        }
        return;
    }
    // this call's epoch for the KV head: one more than the decode calls
    // completed on this workspace (the last kernel of every call advances the
    // device counter), so that a replayed graph of the call still tells the
    // LUT parts' fresh flags from stale ones
    const uint32_t ep = tid < kWave ? counter_read(w.epoch + bg) + 1u : 0u;
    // 1) the samples: runs of kSampleRun positions, rs apart (rs >= 1),
    //    clipped at the next run (short runs: scores within a list
    //    are correlated, so many short runs estimate the quantile with far
    //    less spread than a few long ones). Their codes, norms and lists were
    //    gathered at the index's last prepare or update into one contiguous
    //    slab per KV head: thread tid reads slots u * 512 + tid, one cache
    //    line per 128-byte span instead of one per run and array.
    const SampleRuns sr = sample_runs(n_r);
    const int nrun = sr.nrun;
    const int run_len = sr.run_len;
    const int64_t sbase = static_cast<int64_t>(bg) * kMaxSamples;
    const typename PQ::Code* scodes = reinterpret_cast<const typename PQ::Code*>(ix.samp_codes) + sbase;
    typename PQ::Code cv[kSamplesPer];
    float rv[kSamplesPer];
    int jv[kSamplesPer];
    bool ok[kSamplesPer];
#pragma unroll
    for (int u = 0; u < kSamplesPer; ++u) {
        const int s = u * kProThreads + tid;
        int pos;
        ok[u] = sample_position(sr, s, n_r, pos);
        cv[u] = scodes[s];
        rv[u] = ix.samp_norms[sbase + s];
        jv[u] = ix.samp_list[sbase + s];
    }
    for (int i = tid; i < kHistBins; i += kProThreads) sm.hist[i] = 0;

    // 2) wait for the KV head's LUT parts (bounded): the first wave reads
    //    every part's flag (one per lane, a few cache lines), with two such
    //    reads in flight, spaced out, until all hold this call's epoch
    if (tid < kWave) {
        const int parts = prologue_parts(D.n_list, PQ::BITS);
        const uint32_t* flags = w.lut_flag + bg * parts;
        uint32_t fv[kPolls][kFlagsPerLane];
        auto issue = [&](uint32_t (&f)[kFlagsPerLane]) {
#pragma unroll
            for (int i = 0; i < kFlagsPerLane; ++i)
                f[i] = i * kWave + tid < parts ? counter_read(flags + i * kWave + tid) : ep;
        };
        auto seen = [&](const uint32_t (&f)[kFlagsPerLane]) {
            bool mine = true;
#pragma unroll
            for (int i = 0; i < kFlagsPerLane; ++i) mine = mine && f[i] == ep;
            return __ballot(!mine) == 0ull;
        };
        int ready = 0;
#pragma unroll
        for (int i = 0; i < kPolls; ++i) {
            issue(fv[i]);
            __builtin_amdgcn_s_sleep(kPollSleep);
        }
        for (int it = 0; it < kSpinLimit && !ready; ++it) {
#pragma unroll
            for (int i = 0; i < kPolls; ++i) {
                if (!ready && seen(fv[i])) ready = 1;
                if (!ready) {
                    issue(fv[i]);
                    __builtin_amdgcn_s_sleep(kPollSleep);
                }
            }
        }
        acquire_device();
        if (tid == 0) sm.ready = ready;
    }
    __syncthreads();
    if (!sm.ready) {   // tables not seen in time: every token becomes a candidate
        if (tid == 0) {
            w.tau_lo[row] = neg_inf;
            w.tau_hi[row] = neg_inf;
        }
        return;
    }

    // 3) the head's fine table into LDS, the coarse term of every sample
    constexpr int kLutF4 = (PQ::LUT_ROW / 4 + kProThreads - 1) / kProThreads;   // float4 per thread
    const float4* lsrc = reinterpret_cast<const float4*>(w.lut_head + static_cast<int64_t>(row) * PQ::LUT_ROW);
    float4 lv[kLutF4];
#pragma unroll
    for (int i = 0; i < kLutF4; ++i)
        lv[i] = lsrc[min(i * kProThreads + tid, PQ::LUT_ROW / 4 - 1)];
    const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * G + hh;
    float cf[kSamplesPer];
#pragma unroll
    for (int u = 0; u < kSamplesPer; ++u) cf[u] = coarse[jv[u] * G];
    float4* ldst = reinterpret_cast<float4*>(sm.lut);
#pragma unroll
    for (int i = 0; i < kLutF4; ++i)
        if (i * kProThreads + tid < PQ::LUT_ROW / 4) ldst[i * kProThreads + tid] = lv[i];
    __syncthreads();

    // 4) scores of the samples
    float sc[kSamplesPer];
    uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
    for (int u = 0; u < kSamplesPer; ++u) {
        float fs[1];
        fine_sum<PQ, 1>(sm.lut, cv[u], fs);
        sc[u] = pq_logit(rv[u], cf[u], fs[0]);
        if (ok[u]) {
            const uint32_t kk = float_key(sc[u]);
            mn = min(mn, kk);
            mx = max(mx, kk);
        }
    }
    // their min and max over the workgroup, with one barrier (the scratch is
    // not written again); every run is whole, so there are nrun * run_len
    mn = wave_min_u32(mn);
    mx = wave_max_u32(mx);
    if (lane_id() == 0) {
        sm.bs.v[tid / kWave][0] = mn;
        sm.bs.v[tid / kWave][1] = mx;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kProThreads / kWave; ++i) {
        mn = min(mn, sm.bs.v[i][0]);
        mx = max(mx, sm.bs.v[i][1]);
    }
    const int ns = nrun * run_len;
    // order statistic: about 2k * ns / |R| sampled tokens above, plus a margin
    const int c = (k == 0) ? 1 : static_cast<int>(ceilf(2.0f * k * ns / n_r)) + 8;
    if (c > ns) {   // the budget is a large share of R: every token is a candidate
        if (tid == 0) {
            w.tau_lo[row] = neg_inf;
            w.tau_hi[row] = neg_inf;
        }
        return;
    }
    // 5) bins of equal width in score (monotone: rounded subtraction and
    //    multiplication by a positive constant never reorder two scores)
    const float fmn = key_float(mn);
    const float range = key_float(mx) - fmn;
    const float scale = (range > 0.0f && range < __builtin_huge_valf()) ? kHistBins / range : 0.0f;
#pragma unroll
    for (int u = 0; u < kSamplesPer; ++u) {
        const int bin = min(static_cast<int>((sc[u] - fmn) * scale), kHistBins - 1);
        if (ok[u]) atomicAdd(&sm.hist[bin], 1);   // the samples' bins are mostly distinct
    }
    __syncthreads();
    // 6) one wave: the bin holding the c-th largest sample; tau_lo sits just
    //    below that bin, so at least c samples are >= it
    if (tid < kWave) {
        int above_unused = 0;
        const int bstar = wave_find_bin_desc(sm.hist, c, above_unused);
        if (tid == 0) {
            // the lower edge of the bin below, nudged down: every sample of
            // bin bstar and above (at least c of them) scores at or above it
            // whatever the rounding of the bin computation
            float tl = fmn;
            if (bstar > 1 && scale > 0.0f) {
                tl = fmn + static_cast<float>(bstar - 1) * (range / kHistBins);
                tl = fmaxf(tl - fabsf(tl) * 0x1p-21f, fmn);
            }
            w.tau_lo[row] = tl + bias;
            w.tau_hi[row] = key_float(mx);   // lets the top-k stage fix its bins in advance
        }
    }
}

template <typename T, int G, typename PQ, bool kDev>
__global__ __launch_bounds__(kProThreads) void prologue_kernel(Dims D, BatchArgs ba, Index ix,
                                                               const T* __restrict__ q, Work w,
                                                               float bias, int n_lut_wg) {
    __shared__ SampleLds sm;
    if (static_cast<int>(blockIdx.x) < n_lut_wg) {
        const int per_bg = prologue_parts(D.n_list, PQ::BITS);
        lut_role<T, G, PQ>(D, q, ix.codebooks, ix.centroids, w, blockIdx.x / per_bg,
                           blockIdx.x % per_bg);
        return;
    }
    // sample workgroup s serves group s % NG, head s / NG: workgroups are
    // dispatched to the XCDs round-robin by id, so when the group count is a
    // multiple of 8 the G rows of a group share one L2 and its sample loads
    const int s_idx = blockIdx.x - n_lut_wg;
    const int n_grp = D.B * D.Hkv;
    sample_role<T, G, PQ, kDev>(D, ba, ix, w, bias, (s_idx % n_grp) * G + s_idx / n_grp, sm);
}

template <typename T, int G, typename PQ>
static hipError_t launch_prologue_t(const Dims& D, const BatchArgs& ba, const KV& kv,
                                    const Index& ix, const Work& w, float bias,
                                    hipStream_t s, const KTiming& tm) {
    const int per_bg = prologue_parts(D.n_list, PQ::BITS);
    const int n_lut_wg = D.B * D.Hkv * per_bg;
    const int grid = n_lut_wg + D.B * D.Hq;
    if (w.ba_dev)
        hipExtLaunchKernelGGL((prologue_kernel<T, G, PQ, true>), dim3(grid), dim3(kProThreads), 0, s,
                              tm.start, tm.stop, 0, D, ba, ix, static_cast<const T*>(kv.q), w, bias,
                              n_lut_wg);
    else
        hipExtLaunchKernelGGL((prologue_kernel<T, G, PQ, false>), dim3(grid), dim3(kProThreads), 0, s,
                              tm.start, tm.stop, 0, D, ba, ix, static_cast<const T*>(kv.q), w, bias,
                              n_lut_wg);
    return hipGetLastError();
}

template <typename T, typename PQ>
static hipError_t launch_prologue_g(const Dims& D, const BatchArgs& ba, const KV& kv,
                                    const Index& ix, const Work& w, float bias,
                                    hipStream_t s, const KTiming& tm) {
    switch (D.G) {
        case 1: return launch_prologue_t<T, 1, PQ>(D, ba, kv, ix, w, bias, s, tm);
        case 2: return launch_prologue_t<T, 2, PQ>(D, ba, kv, ix, w, bias, s, tm);
        case 4: return launch_prologue_t<T, 4, PQ>(D, ba, kv, ix, w, bias, s, tm);
        case 8: return launch_prologue_t<T, 8, PQ>(D, ba, kv, ix, w, bias, s, tm);
        default: return hipErrorInvalidValue;
    }
}

template <typename PQ>
static hipError_t launch_prologue_pq(const Dims& D, const BatchArgs& ba, const KV& kv,
                                     const Index& ix, const Work& w, float bias,
                                     hipStream_t s, const KTiming& tm) {
    return kv.bf16 ? launch_prologue_g<bf16_t, PQ>(D, ba, kv, ix, w, bias, s, tm)
                   : launch_prologue_g<float, PQ>(D, ba, kv, ix, w, bias, s, tm);
}

hipError_t launch_prologue(const Dims& D, const BatchArgs& ba, const KV& kv, const Index& ix,
                           const Work& w, float bias, hipStream_t s,
                           const KTiming& tm) {
    return D.pq_bits == 4 ? launch_prologue_pq<Pq4>(D, ba, kv, ix, w, bias, s, tm)
                          : launch_prologue_pq<Pq8>(D, ba, kv, ix, w, bias, s, tm);
}

}  // namespace pqhsa
