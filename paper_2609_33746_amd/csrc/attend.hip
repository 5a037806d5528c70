// Exact attention over E = S u L u T, the per-list background, and the final
// merge (Section 3.2, Eqs. 4-5), plus the dense decode baseline.
//
// Every partial result is a triple (m, Z, N[d]) meaning "sum of
// exp(logit - m) = Z, sum of exp(logit - m) v = N"; partials combine by the
// usual log-sum-exp rule, so the common shift m0 of Section 3.2 never has to
// be known in advance.
//
//  * attend_kernel, exact role: one workgroup per (row, split of kRows rows
//    of E: 64 or 128 by the context's budget). 16 lanes hold one K/V row (8
//    elements each); each 16-lane group owns kRows / 16 rows and issues all
//    of their token-id, K and V
//    loads before any arithmetic, so a workgroup keeps its whole split in
//    flight.
//  * attend_kernel, background role: one workgroup per (batch element, KV
//    head, kBgLists lists). For each list j and each of the G query heads:
//    M_j = (below-threshold mass of the scan segments) * exp(tau_lo - shift)
//          + (weights of the list's unselected candidates from the top-k stage),
//    then Z_B += M_j and N_B += M_j * v_bar_j (Eq. 4), reading each list mean
//    once for the whole group.
//  * merge_kernel: log-sum-exp of all partials of a row, y = N / Z (Eq. 5).
#include "device_common.h"
#include "pqhsa.h"
#include "pqhsa_internal.h"

namespace pqhsa {

constexpr int kAttnThreads = 256;    // 4 waves x 4 groups of 16 lanes = 16 row streams
constexpr int kAttnBgFirstPerCu = 4; // attend grids above this many workgroups per CU put the background first
constexpr int kStreams = kAttnThreads / 16;
// rows per stream in one batch of the dense kernel (two batches are in
// flight; fewer for large groups, which hold G accumulators per lane)
template <int G>
struct DenseBatch { static constexpr int value = G <= 2 ? 4 : 2; };
constexpr int kMergeThreads = kHeadDim;

struct Online {
    float m, z, acc[8];
};

__device__ __forceinline__ void online_init(Online& o) {
    o.m = -__builtin_huge_valf();
    o.z = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) o.acc[t] = 0.0f;
}

// Fold R rows (logits l[i], -inf for absent rows; values v[i]) into o.
template <int R, typename T>
__device__ __forceinline__ void online_push_batch(Online& o, const float (&l)[R],
                                                  const Raw8<T> (&v)[R]) {
    float m_new = o.m;
#pragma unroll
    for (int i = 0; i < R; ++i) m_new = fmaxf(m_new, l[i]);
    if (m_new == -__builtin_huge_valf()) return;   // nothing present yet
    const float a = __expf(o.m - m_new);            // 0 when o.m = -inf
    o.z *= a;
#pragma unroll
    for (int t = 0; t < 8; ++t) o.acc[t] *= a;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const float p = __expf(l[i] - m_new);       // 0 for absent rows
        float x[8];
        v[i].to(x);
        o.z += p;
#pragma unroll
        for (int t = 0; t < 8; ++t) o.acc[t] = fmaf(p, x[t], o.acc[t]);
    }
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
#pragma unroll
        for (int s = 0; s < kStreams; ++s) M = fmaxf(M, sm[s]);
        float Z = 0.0f, N = 0.0f;
        if (M != -__builtin_huge_valf()) {
#pragma unroll
            for (int s = 0; s < kStreams; ++s) {
                const float f = __expf(sm[s] - M);
                Z = fmaf(sz[s], f, Z);
                N = fmaf(sacc[s * kHeadDim + t], f, N);
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

// kBx: variant Bx. The exact role subtracts, at the background's shift, the
// selected rows weighted by their lists' W_j = M_j / |B n R_j|; the background
// role weights list j's mean by W_j |R_j| instead of M_j.
template <typename T, int G, bool kBx, bool kDev, int kRows>
__global__ __launch_bounds__(kAttnThreads) void attend_kernel(Dims D, BatchArgs ba, KV kv,
                                                              Index ix, Work w, int nsplit,
                                                              int nsplit_max, int n_bgc,
                                                              int variant, int bg_first) {
    constexpr int kRowsPerStream = kRows / kStreams;
    __shared__ float sm[kStreams], sz[kStreams];
    // [16 streams][d] for the exact role, [4 waves][G][d] for the background role
    __shared__ float sacc[(kStreams > 4 * G ? kStreams : 4 * G) * kHeadDim];
    __shared__ float bz[4][G];
    const int n_exact_wg = D.B * D.Hq * nsplit;
    const int n_bg_wg = variant == PQHSA_VARIANT_T ? 0 : D.B * D.Hkv * n_bgc;
    const int first_exact = bg_first ? n_bg_wg : 0;      // grid order of the two roles
    const int first_bg = bg_first ? 0 : n_exact_wg;
    const int P = nsplit_max + n_bgc;
    const int lane16 = threadIdx.x & 15;
    const int stream = threadIdx.x >> 4;
    const float neg_inf = -__builtin_huge_valf();

    const int xid = static_cast<int>(blockIdx.x) - first_exact;
    if (xid >= 0 && xid < n_exact_wg) {
        // ---------------- exact attention over a split of E ----------------
        const int row = xid / nsplit;
        const int split = xid % nsplit;
        const int b = row / D.Hq;
        const int h = row % D.Hq;
        const int g = h / G;
        const int k = arg_topk<kDev>(ba, w, b);
        const int n_r = arg_n_r<kDev>(ba, w, b);
        const int n_tail = arg_n_tail<kDev>(ba, w, b);   // L_b = [n_sink + |R_b|, N_b)
        const int nE = D.n_sink + n_tail + k;
        const int e0 = split * kRows;
        if (e0 >= nE) return;   // the merge reads only the splits that exist
        const int e1 = min(e0 + kRows, nE);
        const int32_t* sel = w.sel_tok + static_cast<int64_t>(row) * D.max_topk;
        const int local0 = D.n_sink + n_r;
        int tok[kRowsPerStream];
#pragma unroll
        for (int i = 0; i < kRowsPerStream; ++i) {
            const int e = e0 + stream + i * kStreams;
            int t = -1;
            if (e < e1) {
                if (e < D.n_sink) t = e;
                else if (e < D.n_sink + n_tail) t = local0 + (e - D.n_sink);
                else t = min(max(sel[e - D.n_sink - n_tail], D.n_sink), local0 - 1);   // never outside R
            }
            tok[i] = t;
        }
        float wx[kRowsPerStream];   // Bx: W of the row's list for rows of T, else 0
        float bx_shift = neg_inf;
        if constexpr (kBx) {
            const float* wsel = w.bx_wsel + static_cast<int64_t>(row) * D.max_topk;
#pragma unroll
            for (int i = 0; i < kRowsPerStream; ++i) {
                const int e = e0 + stream + i * kStreams;
                wx[i] = e < e1 && e >= D.n_sink + n_tail ? wsel[e - D.n_sink - n_tail] : 0.0f;
            }
            bx_shift = w.row_shift[row];
        }
        const T* kb = static_cast<const T*>(kv.k) + lane16 * 8;
        const T* vb = static_cast<const T*>(kv.v) + lane16 * 8;
        int64_t roff[kRowsPerStream];   // a paged cache adds one block-table read
#pragma unroll
        for (int i = 0; i < kRowsPerStream; ++i) roff[i] = tok[i] >= 0 ? kv_row(kv, b, g, tok[i]) : 0;
        Raw8<T> kr[kRowsPerStream], vr[kRowsPerStream];
#pragma unroll
        for (int i = 0; i < kRowsPerStream; ++i) {
            if (tok[i] >= 0) {
                kr[i].load(kb + roff[i]);
                vr[i].load(vb + roff[i]);
            } else {
                kr[i].zero();
                vr[i].zero();
            }
        }
        float qv[8];
        Load8<T>::run(static_cast<const T*>(kv.q) + static_cast<int64_t>(row) * kHeadDim + lane16 * 8, qv);
        float l[kRowsPerStream];
#pragma unroll
        for (int i = 0; i < kRowsPerStream; ++i) {
            float kf[8];
            kr[i].to(kf);
            float dot = 0.0f;
#pragma unroll
            for (int t = 0; t < 8; ++t) dot = fmaf(qv[t], kf[t], dot);
            dot = sum16(dot);
            l[i] = tok[i] >= 0 ? dot * D.inv_sqrt_d : neg_inf;
        }
        Online o;
        online_init(o);
        online_push_batch<kRowsPerStream>(o, l, vr);
        if constexpr (kBx) {
            // fold -sum_i W_i v_i, which lives at the background's shift, into
            // the stream's state under m' = max(m, shift) (both factors <= 1)
            if (bx_shift != neg_inf) {
                float c[8] = {};
#pragma unroll
                for (int i = 0; i < kRowsPerStream; ++i) {
                    float x[8];
                    vr[i].to(x);
#pragma unroll
                    for (int t = 0; t < 8; ++t) c[t] = fmaf(wx[i], x[t], c[t]);
                }
                const float m2 = fmaxf(o.m, bx_shift);
                const float a = __expf(o.m - m2);   // 0 when o.m = -inf
                const float f = __expf(bx_shift - m2);
                o.z *= a;
#pragma unroll
                for (int t = 0; t < 8; ++t) o.acc[t] = fmaf(o.acc[t], a, -c[t] * f);
                o.m = m2;
            }
        }
        block_combine(o, sm, sz, sacc,
                      w.partial + (static_cast<int64_t>(row) * P + split) * kPartStride);
        return;
    }

    // ---------------- per-list background (Eq. 4) ----------------
    const int idx = static_cast<int>(blockIdx.x) - first_bg;
    const int bg = idx / n_bgc;
    const int lc = idx % n_bgc;
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;
    const int row0 = b * D.Hq + g * G;
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    constexpr int kWaves = kAttnThreads / kWave;
    constexpr int kListsPerWave = kBgLists / kWaves;   // 16

    // lanes 0..15 each compute the masses M_j of one list of this wave:
    // M_j = (scan segments below tau_lo) * exp(tau_lo - shift)
    //       + (unselected candidates of list j, already relative to shift);
    // the segments of list l & 15 are summed by the four lanes l, l + 16,
    // l + 32 and l + 48, each taking every fourth one, so a long list costs
    // a quarter of the loads per lane (a 64-list workgroup ends with its
    // longest list)
    constexpr int kSegLanes = kWave / kListsPerWave;   // 4
    static_assert(kSegLanes * kListsPerWave == kWave && kSegLanes == 4, "four lanes per list");
    const int seg_q = lane / kListsPerWave;
    const int my_j = lc * kBgLists + wave + (lane & (kListsPerWave - 1)) * kWaves;
    // every load that does not depend on another is issued first: the list
    // offsets (first, since a wave's loads return in order and the segment
    // loads wait for them), the list means and the candidate weights; then
    // the list's scan segments. The rows' shifts and thresholds (scalar
    // loads) come after, so that no vector load waits behind them.
    const bool okj = my_j < D.n_list;
    const int jj = okj ? my_j : 0;
    const int32_t* loff = ix.loff + static_cast<int64_t>(bg) * (D.n_list + 1);
    const int lo = loff[jj];
    const int hi = okj ? loff[jj + 1] : lo;
    // variant C: every list takes the global value mean of R_b
    const bool global_mean = variant == PQHSA_VARIANT_C;
    float2 vbar[kListsPerWave];
#pragma unroll
    for (int i = 0; i < kListsPerWave; ++i) {
        const int j = lc * kBgLists + wave + i * kWaves;
        const float* src = global_mean
                               ? ix.glob_mean + static_cast<int64_t>(bg) * kHeadDim
                               : ix.means + (static_cast<int64_t>(bg) * D.n_list + j) * kHeadDim;
        vbar[i] = j < D.n_list ? *reinterpret_cast<const float2*>(src + 2 * lane)
                               : make_float2(0.f, 0.f);
    }
    float mj[G], mn[G];   // M_j, and the weight of v_bar_j in N (M_j, or W_j |R_j| for Bx)
    float shift[G], below_scale[G];
    bool live[G];
    {
        const bool ok = seg_q == 0 && okj;
        float cand[G];
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
            cand[hh] = ok ? w.cand_mass[static_cast<int64_t>(row0 + hh) * D.n_list + jj] : 0.0f;
        // list j's positions [lo, hi) span sub-chunks lo / kSub .. (hi - 1) / kSub,
        // whose masses sit at segments j + s
        const int s0 = jj + lo / kSub;
        const int s1 = hi > lo ? jj + (hi - 1) / kSub + 1 : s0;
        const float* segs = w.seg_sum + static_cast<int64_t>(bg) * D.nseg_cap * G;
        // this lane's segments s0 + seg_q + 4 i, kSegsAtOnce per round trip
        constexpr int kSegsAtOnce = 2;
        float below[G];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) below[hh] = 0.0f;
        for (int s = s0 + seg_q; s < s1; s += kSegLanes * kSegsAtOnce) {
            float sv[kSegsAtOnce][G];
#pragma unroll
            for (int u = 0; u < kSegsAtOnce; ++u)
#pragma unroll
                for (int hh = 0; hh < G; ++hh)
                    sv[u][hh] = s + kSegLanes * u < s1 ? segs[(s + kSegLanes * u) * G + hh] : 0.0f;
#pragma unroll
            for (int u = 0; u < kSegsAtOnce; ++u)
#pragma unroll
                for (int hh = 0; hh < G; ++hh) below[hh] += sv[u][hh];
        }
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            below[hh] += __shfl_xor(below[hh], kListsPerWave);
            below[hh] += __shfl_xor(below[hh], 2 * kListsPerWave);
        }
        // the rows' shifts and thresholds, read after every vector load is out
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            shift[hh] = w.row_shift[row0 + hh];
            const float tlo = w.tau_lo[row0 + hh];
            live[hh] = shift[hh] != neg_inf;
            const bool use_below = live[hh] && tlo != neg_inf && w.row_flag[row0 + hh] == 0;
            below_scale[hh] = use_below ? __expf(tlo - shift[hh]) : 0.0f;
        }
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            mj[hh] = (ok && live[hh]) ? below[hh] * below_scale[hh] + cand[hh] : 0.0f;
            mn[hh] = mj[hh];
            if constexpr (kBx)
                mn[hh] = (ok && live[hh])
                             ? w.bx_w[static_cast<int64_t>(row0 + hh) * D.n_list + jj] * static_cast<float>(hi - lo)
                             : 0.0f;
        }
    }
    float Z[G], N[G][2];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) { Z[hh] = 0.0f; N[hh][0] = 0.0f; N[hh][1] = 0.0f; }
#pragma unroll
    for (int i = 0; i < kListsPerWave; ++i) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            const float Mj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mj[hh]), i));
            const float Mn = kBx ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mn[hh]), i)) : Mj;
            Z[hh] += Mj;
            N[hh][0] = fmaf(Mn, vbar[i].x, N[hh][0]);
            N[hh][1] = fmaf(Mn, vbar[i].y, N[hh][1]);
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
// Partials [0, n_exact(b)) and [first_bg, first_bg + n_bg) of each row are used;
// partials with Z = 0 are skipped. Per batch of kMergeBatch used partials,
// thread u < kMergeBatch loads (m, Z) of partial u and every thread t loads
// N[t] of all of them, all at once, so a row with at most kMergeBatch
// partials costs one memory round trip; batches fold by the log-sum-exp rule.
constexpr int kMergeBatch = 40;
static_assert(kMergeBatch <= kMergeThreads, "one (m, Z) per thread");

// kGroups groups of kMergeThreads threads: group gi folds batches gi,
// gi + kGroups, ... of the row's partials, then the groups' results fold in
// LDS. One group serves rows of up to kMergeBatch (40) partials and two
// groups rows of up to 80, each in one round trip (the PQ-HSA rows and the
// dense decode up to 128K rows); longer dense rows (more than 80 splits of
// 2048 rows) take 8. (40 partials per group: a 128K row of 64-row splits has
// 39; the merge took 4.3 us against 4.8 us with two groups of 32.)
template <int kGroups>
__global__ __launch_bounds__(kMergeThreads * kGroups) void merge_kernel(
    Dims D, BatchInts n_exact_parts, const float* __restrict__ partial, int P, int first_bg,
    int n_bg, float* __restrict__ out, uint32_t* epoch, const BatchArgs* ba_dev) {
    // the decode call is complete once this launch is: the first row of each
    // (batch element, KV head) advances the epoch the next call's prologue
    // reads for it (the dense decode passes none)
    if (epoch && threadIdx.x == 0 && (blockIdx.x % D.Hq) % D.G == 0)
        counter_add(epoch + blockIdx.x / D.Hq * D.Hkv + (blockIdx.x % D.Hq) / D.G, 1u);
    __shared__ float2 smz[kGroups][kMergeBatch];
    __shared__ float gm[kGroups], gz[kGroups];
    __shared__ float gn[kGroups > 1 ? kGroups : 1][kMergeThreads];
    const int row = blockIdx.x;
    const int b = row / D.Hq;
    const int gi = kGroups > 1 ? static_cast<int>(threadIdx.x) / kMergeThreads : 0;
    const int t = kGroups > 1 ? static_cast<int>(threadIdx.x) % kMergeThreads : static_cast<int>(threadIdx.x);
    const float* pr = partial + static_cast<int64_t>(row) * P * kPartStride;
    // exact partials of the row: from the host, or from the call's device
    // budgets and lengths
    const int ne = ba_dev ? (D.n_sink + ba_dev->n_tail[b] + ba_dev->topk[b] + D.attn_rows - 1) / D.attn_rows
                          : n_exact_parts.v[b];
    const int n_used = ne + n_bg;
    const float neg_inf = -__builtin_huge_valf();
    auto part = [&](int i) { return i < ne ? i : first_bg + (i - ne); };   // i-th used partial
    float M = neg_inf, Z = 0.0f, N = 0.0f;
    for (int r0 = 0; r0 < n_used; r0 += kGroups * kMergeBatch) {   // the same trip count in every group
        const int i0 = r0 + gi * kMergeBatch;
        float2 mz = make_float2(neg_inf, 0.0f);
        if (t < kMergeBatch && i0 + t < n_used)
            mz = *reinterpret_cast<const float2*>(pr + part(i0 + t) * kPartStride);
        float n[kMergeBatch];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u)
            n[u] = i0 + u < n_used ? pr[part(i0 + u) * kPartStride + 4 + t] : 0.0f;
        if (t < kMergeBatch) smz[gi][t] = mz.y > 0.0f ? mz : make_float2(neg_inf, 0.0f);
        __syncthreads();
        float mb = M;
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) mb = fmaxf(mb, smz[gi][u].x);
        if (mb != neg_inf) {
            const float a = __expf(M - mb);   // 0 while M = -inf
            Z *= a;
            N *= a;
#pragma unroll
            for (int u = 0; u < kMergeBatch; ++u) {
                const float2 e = smz[gi][u];
                const float f = e.x == neg_inf ? 0.0f : __expf(e.x - mb);
                Z = fmaf(e.y, f, Z);
                N = f != 0.0f ? fmaf(n[u], f, N) : N;
            }
            M = mb;
        }
        __syncthreads();
    }
    if constexpr (kGroups > 1) {
        if (t == 0) {
            gm[gi] = M;
            gz[gi] = Z;
        }
        gn[gi][t] = N;
        __syncthreads();
        if (gi != 0) return;
        float mt = neg_inf;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) mt = fmaxf(mt, gm[g]);
        Z = 0.0f;
        N = 0.0f;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            const float f = gm[g] == neg_inf ? 0.0f : __expf(gm[g] - mt);
            Z = fmaf(gz[g], f, Z);
            N = fmaf(gn[g][t], f, N);
        }
    }
    out[static_cast<int64_t>(row) * kHeadDim + t] = N / Z;
}

template <typename T, int G, bool kDev>
static hipError_t launch_attend_d(const Dims& D, const BatchArgs& ba, const KV& kv,
                                  const Index& ix, const Work& w, int nsplit, int nsplit_max,
                                  int variant, hipStream_t s, const KTiming& tm) {
    const int n_bgc = (D.n_list + kBgLists - 1) / kBgLists;   // the partials' layout
    // variant T has no background: the background workgroups are not launched
    const int grid = D.B * D.Hq * nsplit + (variant == PQHSA_VARIANT_T ? 0 : D.B * D.Hkv * n_bgc);
    // Beyond about one round of resident workgroups, the background workgroups
    // (the longer chain of loads) go first, so that they do not start only
    // after every exact workgroup: 4 sequences at 128K, 40.7 -> 39.4 us. In a
    // single round the exact ones go first (0.3 us better at one sequence).
    const int bg_first = grid > kAttnBgFirstPerCu * device_cu_count() ? 1 : 0;
    auto kern = variant == PQHSA_VARIANT_BX
                    ? (D.attn_rows == kAttnRowsSmall ? attend_kernel<T, G, true, kDev, kAttnRowsSmall>
                                                     : attend_kernel<T, G, true, kDev, kAttnRows>)
                    : (D.attn_rows == kAttnRowsSmall ? attend_kernel<T, G, false, kDev, kAttnRowsSmall>
                                                     : attend_kernel<T, G, false, kDev, kAttnRows>);
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(kAttnThreads), 0, s, tm.start, tm.stop, 0, D, ba, kv,
                          ix, w, nsplit, nsplit_max, n_bgc, variant, bg_first);
    return hipGetLastError();
}

template <typename T, int G>
static hipError_t launch_attend_t(const Dims& D, const BatchArgs& ba, const KV& kv,
                                  const Index& ix, const Work& w, int nsplit, int nsplit_max,
                                  int variant, hipStream_t s, const KTiming& tm) {
    return w.ba_dev ? launch_attend_d<T, G, true>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm)
                    : launch_attend_d<T, G, false>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm);
}

template <typename T>
static hipError_t launch_attend_g(const Dims& D, const BatchArgs& ba, const KV& kv,
                                  const Index& ix, const Work& w, int nsplit, int nsplit_max,
                                  int variant, hipStream_t s, const KTiming& tm) {
    switch (D.G) {
        case 1: return launch_attend_t<T, 1>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm);
        case 2: return launch_attend_t<T, 2>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm);
        case 4: return launch_attend_t<T, 4>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm);
        case 8: return launch_attend_t<T, 8>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attend(const Dims& D, const BatchArgs& ba, const KV& kv, const Index& ix,
                         const Work& w, int nsplit, int nsplit_max, int variant, hipStream_t s,
                         const KTiming& tm) {
    return kv.bf16 ? launch_attend_g<bf16_t>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm)
                   : launch_attend_g<float>(D, ba, kv, ix, w, nsplit, nsplit_max, variant, s, tm);
}

static hipError_t launch_merge_parts(const Dims& D, const BatchInts& ne, const float* partial,
                                     int P, int first_bg, int n_bg, float* out, uint32_t* epoch,
                                     const BatchArgs* ba_dev, hipStream_t s, const KTiming& tm) {
    int most = 0;   // the most partials of a row
    for (int b = 0; b < D.B; ++b) most = ne.v[b] + n_bg > most ? ne.v[b] + n_bg : most;
    // one memory round trip per row: one group of threads per batch of
    // kMergeBatch partials (up to 2), or 8 groups looping for the dense rows
    if (most <= kMergeBatch)
        hipExtLaunchKernelGGL(merge_kernel<1>, dim3(D.B * D.Hq), dim3(kMergeThreads), 0, s, tm.start,
                              tm.stop, 0, D, ne, partial, P, first_bg, n_bg, out, epoch, ba_dev);
    else if (most <= 2 * kMergeBatch)
        hipExtLaunchKernelGGL(merge_kernel<2>, dim3(D.B * D.Hq), dim3(2 * kMergeThreads), 0, s,
                              tm.start, tm.stop, 0, D, ne, partial, P, first_bg, n_bg, out, epoch, ba_dev);
    else
        hipExtLaunchKernelGGL(merge_kernel<8>, dim3(D.B * D.Hq), dim3(8 * kMergeThreads), 0, s,
                              tm.start, tm.stop, 0, D, ne, partial, P, first_bg, n_bg, out, epoch, ba_dev);
    return hipGetLastError();
}

hipError_t launch_merge(const Dims& D, const BatchArgs& ba, const Work& w, float* out,
                        int nsplit_max, int variant, hipStream_t s, const KTiming& tm) {
    BatchInts ne;
    for (int b = 0; b < D.B; ++b) {
        // with device budgets the kernel counts the partials itself; the
        // bound here only picks the launch shape
        const int nE = D.n_sink + ba.n_tail[b] + ba.topk[b];
        ne.v[b] = w.ba_dev ? nsplit_max : (nE + D.attn_rows - 1) / D.attn_rows;
    }
    const int n_bgc = (D.n_list + kBgLists - 1) / kBgLists;
    // variant T: the exact partials alone
    return launch_merge_parts(D, ne, w.partial, nsplit_max + n_bgc, nsplit_max,
                              variant == PQHSA_VARIANT_T ? 0 : n_bgc, out, w.epoch, w.ba_dev, s, tm);
}

// ---------------------------------------------------------------------------
// Dense decode baseline: every cached row, all G heads of a group per K/V load.
// Each 16-lane stream walks rows stream, stream + 16, ... of its split; the
// loads of the next batch of rows are issued before the current batch is
// used, so every stream keeps two batches in flight. bf16 queries stay packed
// and the q.k products use the two-way bf16 dot instruction (fp32 sums).
// ---------------------------------------------------------------------------
template <typename T, int G>
struct DenseQ;

template <int G>
struct DenseQ<bf16_t, G> {
    uint32_t q[G][4];
    __device__ __forceinline__ void load(const bf16_t* p, int64_t head_stride) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            const uint4 w = *reinterpret_cast<const uint4*>(p + hh * head_stride);
            q[hh][0] = w.x; q[hh][1] = w.y; q[hh][2] = w.z; q[hh][3] = w.w;
        }
    }
    __device__ __forceinline__ float dot(int hh, const Raw8<bf16_t>& k) const {
        const uint32_t kw[4] = {k.w.x, k.w.y, k.w.z, k.w.w};
        float d = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) d = dot2_bf16(q[hh][i], kw[i], d);
        return d;
    }
};

template <int G>
struct DenseQ<float, G> {
    float q[G][8];
    __device__ __forceinline__ void load(const float* p, int64_t head_stride) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh) Load8<float>::run(p + hh * head_stride, q[hh]);
    }
    __device__ __forceinline__ float dot(int hh, const Raw8<float>& k) const {
        float kf[8];
        k.to(kf);
        float d = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d = fmaf(q[hh][e], kf[e], d);
        return d;
    }
};

template <typename T, int R>
__device__ __forceinline__ void dense_load(Raw8<T> (&kr)[R], Raw8<T> (&vr)[R], const T* kb,
                                           const T* vb, int64_t sn, int base, int t1) {
    // rows past t1 re-read row t1 - 1 (their logits are masked to -inf, so
    // their weights are exactly 0): no branch around the loads
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t t = min(base + i * kStreams, t1 - 1);
        kr[i].load(kb + t * sn);
        vr[i].load(vb + t * sn);
    }
}

// Fold R rows into o with a lazily moved shift: o.m changes only when a row's
// logit exceeds it by more than kLazyShift, so the weights exp(l - o.m) stay
// below e^kLazyShift (far from fp32 overflow) and the rescaling of the
// accumulators, the costliest part of a fold, is skipped for almost every
// batch. The result equals the eager fold up to rounding.
constexpr float kLazyShift = 8.0f;
template <int R, typename T>
__device__ __forceinline__ void online_push_lazy(Online& o, const float (&l)[R],
                                                 const Raw8<T> (&v)[R]) {
    float m_new = l[0];
#pragma unroll
    for (int i = 1; i < R; ++i) m_new = fmaxf(m_new, l[i]);
    if (m_new > o.m + kLazyShift) {   // also the first present row (o.m = -inf)
        const float a = __expf(o.m - m_new);   // 0 when o.m = -inf
        o.z *= a;
#pragma unroll
        for (int t = 0; t < 8; ++t) o.acc[t] *= a;
        o.m = m_new;
    }
    if (o.m == -__builtin_huge_valf()) return;   // nothing present yet
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const float p = __expf(l[i] - o.m);   // 0 for absent rows
        float x[8];
        v[i].to(x);
        o.z += p;
#pragma unroll
        for (int t = 0; t < 8; ++t) o.acc[t] = fmaf(p, x[t], o.acc[t]);
    }
}

// Fold rows base, base + 16, ... (R of them; those at or past t1 are absent)
// into the G heads' online states.
template <typename T, int G, int R>
__device__ __forceinline__ void dense_rows(const DenseQ<T, G>& qv, Online (&o)[G],
                                           const Raw8<T> (&kr)[R], const Raw8<T> (&vr)[R],
                                           int base, int t1, float inv_sqrt_d) {
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        float l[R];
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const float dot = sum16(qv.dot(hh, kr[i]));
            l[i] = base + i * kStreams < t1 ? dot * inv_sqrt_d : -__builtin_huge_valf();
        }
        online_push_lazy<R>(o[hh], l, vr);
    }
}

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
    DenseQ<T, G> qv;
    qv.load(static_cast<const T*>(kv.q) + (static_cast<int64_t>(b) * D.Hq + g * G) * kHeadDim +
                lane16 * 8,
            kHeadDim);
    const T* kb = static_cast<const T*>(kv.k) + b * kv.sb + g * kv.sh + lane16 * 8;
    const T* vb = static_cast<const T*>(kv.v) + b * kv.sb + g * kv.sh + lane16 * 8;
    Online o[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) online_init(o[hh]);
    constexpr int R = DenseBatch<G>::value;
    constexpr int kStep = kStreams * R;
    // two register sets take turns: one is being loaded while the other is used
    Raw8<T> ka[R], va[R], kc[R], vc[R];
    dense_load<T, R>(ka, va, kb, vb, kv.sn, t0 + stream, t1);
    for (int base = t0 + stream; base < t1; base += 2 * kStep) {
        dense_load<T, R>(kc, vc, kb, vb, kv.sn, base + kStep, t1);
        dense_rows<T, G, R>(qv, o, ka, va, base, t1, D.inv_sqrt_d);
        if (base + kStep >= t1) break;
        dense_load<T, R>(ka, va, kb, vb, kv.sn, base + 2 * kStep, t1);
        dense_rows<T, G, R>(qv, o, kc, vc, base + kStep, t1, D.inv_sqrt_d);
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
    return launch_merge_parts(D, ne, partial, nsplit_max, 0, 0, out, nullptr, nullptr, s, KTiming{});
}

}  // namespace pqhsa
