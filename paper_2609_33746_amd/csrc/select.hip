// Top-k selection (Section 3.2, Eq. 3): T = the k indexed tokens with the
// largest approximate logits, per (batch element, query head) row, ties to the
// smaller token id.
//
// One workgroup per row gathers the row's candidates (the tokens the scan
// found at or above the sampled threshold tau_lo, in list-major position
// order) into LDS, locates the k-th largest score with one histogram pass
// over monotone bins of the order keys, ranks the few candidates of the
// boundary bin exactly (score, then token id), writes T, and sums
// exp(l~ - shift) of the unselected candidates per list (in 64-bit fixed
// point, so the sums do not depend on the order of the atomic additions).
// If the threshold left fewer than k candidates (or none at all), the row is
// re-scanned in full from the LUT and every indexed token becomes a
// candidate; the below-threshold masses of the scan are then ignored for that
// row. Rows with more candidates than the LDS holds, or a very dense boundary
// bin, use a radix select instead. Every path gives the exact top-k.
//
// Each wave loads the counts of its own sub-chunks and scans them with DPP,
// candidate loads are issued in batches, and every workgroup-wide step is one
// scan or reduction, so the dependency chain stays short.
#include <type_traits>

#include "device_common.h"
#include "hist_select.h"
#include "pq_score.h"
#include "pqhsa_internal.h"
#include "radix_select.h"

namespace pqhsa {

constexpr int kNW = kSelThreads / kWave;
constexpr int kRankCap = 128;
constexpr int kNzSubBits = 10;           // sub-chunk bits of a nonempty-list entry
static_assert((1 << kNzSubBits) >= kSelMaxSub, "sub-chunk ids");
static_assert(kSelCap < (1 << (31 - kNzSubBits)), "first-candidate indices");          // boundary-bin keys ranked exactly (O(m^2 / 64) ballots)
constexpr float kMassScale = 1099511627776.0f;       // 2^40: fixed-point weights
constexpr float kMassUnscale = 1.0f / 1099511627776.0f;

// Bin of a key under bins fixed before the candidates are seen: keys from
// bkmin upward in steps of 2^bsh, everything above the last bin in it.
__device__ __forceinline__ uint32_t fixed_bin(uint32_t key, uint32_t bkmin, int bsh) {
    return key >= bkmin ? min((key - bkmin) >> bsh, static_cast<uint32_t>(kHistBins - 1)) : 0u;
}

// Rank the keys of one histogram bin exactly: key desc, then token id asc.
// The bin's keys are gathered into r_key / r_idx, then each wave ranks some of
// them against all the others with one ballot per 64 keys; token ids
// (tok_at) are read only when two keys of the bin are equal. Marks the `need`
// largest in the `chosen` bitmap and returns the need-th largest key in kth.
// Returns false without marking anything when the bin holds more than
// kRankCap keys. Must be called by the whole workgroup; flags[0] must be 0.
template <typename KeyAt, typename TokAt>
__device__ __forceinline__ bool rank_boundary_bin(KeyAt key_at, TokAt tok_at, int n, uint32_t kmin,
                                                  int sh, int bin, int m, int need, uint32_t* r_key,
                                                  int* r_idx, int* r_tok, int* counter, int* flags,
                                                  uint32_t* chosen, uint32_t& kth,
                                                  BlockScratch& bs) {
    if (m > kRankCap) return false;
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = lane_id();
    for (int i0 = 0; i0 < n; i0 += kSelThreads) {
        const int i = i0 + tid;
        if (i < n) {
            const uint32_t kk = key_at(i);
            if (static_cast<int>(fixed_bin(kk, kmin, sh)) == bin) {
                const int slot = atomicAdd(counter, 1);
                r_key[slot] = kk;
                r_idx[slot] = i;
            }
        }
    }
    __syncthreads();
    // pass 1: rank by key alone, and look for equal keys
    for (int i = wave; i < m; i += kNW) {
        const uint32_t ki = r_key[i];
        int rank = 0;
        bool dup = false;
        for (int j0 = 0; j0 < m; j0 += kWave) {
            const int j = j0 + lane;
            const uint32_t kj = j < m ? r_key[j] : 0u;
            rank += __popcll(__ballot(j < m && kj > ki));
            dup |= __ballot(j < m && j != i && kj == ki) != 0ull;
        }
        if (dup) {
            if (lane == 0) flags[0] = 1;
        } else if (lane == 0 && rank < need) {
            const int idx = r_idx[i];
            atomicOr(&chosen[idx >> 5], 1u << (idx & 31));
            if (rank == need - 1) bs.bcast[2] = static_cast<int>(ki);
        }
    }
    __syncthreads();
    if (flags[0]) {
        // equal keys in the bin: rank again with the token ids
        if (tid < m) r_tok[tid] = tok_at(r_idx[tid]);
        __syncthreads();
        for (int i = wave; i < m; i += kNW) {
            const uint32_t ki = r_key[i];
            const int ti = r_tok[i];
            int rank = 0;
            bool dup = false;
            for (int j0 = 0; j0 < m; j0 += kWave) {
                const int j = j0 + lane;
                const uint32_t kj = j < m ? r_key[j] : 0u;
                const int tj = j < m ? r_tok[j] : 0;
                rank += __popcll(__ballot(j < m && (kj > ki || (kj == ki && tj < ti))));
                dup |= __ballot(j < m && j != i && kj == ki) != 0ull;
            }
            // keys that had no equal were marked by pass 1 already
            if (dup && lane == 0 && rank < need) {
                const int idx = r_idx[i];
                atomicOr(&chosen[idx >> 5], 1u << (idx & 31));
            }
            if (lane == 0 && rank == need - 1) bs.bcast[2] = static_cast<int>(ki);
        }
        __syncthreads();
    }
    kth = static_cast<uint32_t>(bs.bcast[2]);
    __syncthreads();
    return true;
}

// LDS layout of select_kernel (dynamic, 4-byte words), for kCap candidates:
//   keys [kCap] | cand [kCap] | hist [kHistBins] | rank_key [kRankCap] |
//   rank_idx [kRankCap] | rank_tok [kRankCap] | chosen bitmap [kCap / 32] |
//   counter, flags [4] | sub-chunk offsets, or the nonempty sub-chunks, [kSelMaxSub] |
//   mass (uint64) [n_list]
template <int kCap>
struct SelLayout {
    static constexpr int kOffCand = kCap;
    static constexpr int kOffHist = 2 * kCap;
    static constexpr int kOffRKey = kOffHist + kHistBins;
    static constexpr int kOffRIdx = kOffRKey + kRankCap;
    static constexpr int kOffRTok = kOffRIdx + kRankCap;
    static constexpr int kOffBits = kOffRTok + kRankCap;
    static constexpr int kOffCounter = kOffBits + kCap / 32;
    static constexpr int kOffSub = kOffCounter + 4;
    static constexpr int kOffMass = (kOffSub + kSelMaxSub + 1) & ~1;   // 8-byte aligned
    static size_t bytes(int n_list) { return static_cast<size_t>(kOffMass + 2 * n_list) * 4; }
    static_assert(kCap % kSelThreads == 0 && kCap % 32 == 0, "whole copy tiers and bitmap words");
    static_assert(kOffCand % 4 == 0, "16-byte candidate stores");
};
// Two capacities: every row's candidates of a large budget in LDS (one
// workgroup per CU), or fewer (two workgroups per CU, for grids of more rows
// than CUs; rows beyond it take the global-memory path).
constexpr int kSelCapSmall = 7168;

// Copy the row's `total` candidates (1 <= total <= N * kSelThreads) from
// their sub-chunk slots into LDS in position order (one workgroup per CU): keys at lds[i], words
// (list << kPosBits | token) at lds[kOffCand + i]. Thread t copies the
// indices u * kSelThreads + t, so neighbouring lanes read neighbouring
// slots. Candidate i lives in the sub-chunk sc with pre[sc] <= i < pre[sc + 1]
// (the last of equal offsets, so empty sub-chunks never match). Every thread
// searches all of its indices together and issues all loads before using
// any, so the copy costs one search chain and one memory round trip
// (indices past the end repeat the last candidate's load). Tracks this
// thread's min / max key.
// With fixed bins (hist != nullptr), every candidate is also counted in
// hist at bin min((key - bkmin) >> bsh, kHistBins - 1).
template <int N, int kOffCand>
__device__ __forceinline__ void copy_candidates_search(const uint2* __restrict__ cand, const int* pre,
                                                int nsub, int total, uint32_t* lds,
                                                uint32_t& kmin, uint32_t& kmax, int* hist,
                                                uint32_t bkmin, int bsh) {
    const int tid = threadIdx.x;
    // the N searches advance together, one step at a time, so their LDS
    // reads overlap instead of forming one long dependent chain
    int cs[N], ci[N];
#pragma unroll
    for (int u = 0; u < N; ++u) {
        ci[u] = min(u * kSelThreads + tid, total - 1);
        cs[u] = 0;
    }
#pragma unroll
    for (int step = kSelMaxSub / 2; step > 0; step >>= 1) {
        int pv[N];
#pragma unroll
        for (int u = 0; u < N; ++u) pv[u] = pre[min(cs[u] + step, kSelMaxSub - 1)];
#pragma unroll
        for (int u = 0; u < N; ++u) {
            const int t = cs[u] + step;
            if (t < nsub && pv[u] <= ci[u]) cs[u] = t;
        }
    }
    uint2 rec[N];
#pragma unroll
    for (int u = 0; u < N; ++u) {
        const int slot = min(u * kSelThreads + tid, total - 1) - pre[cs[u]];   // in [0, count)
        rec[u] = cand[static_cast<int64_t>(cs[u]) * kSub + slot];
    }
#pragma unroll
    for (int u = 0; u < N; ++u) {
        const int ci = u * kSelThreads + tid;
        const uint32_t kk = float_key(__uint_as_float(rec[u].x));
        if (ci < total) {
            lds[ci] = kk;
            lds[kOffCand + ci] = rec[u].y;
            kmin = min(kmin, kk);
            kmax = max(kmax, kk);
        }
        // one LDS atomic per candidate: their bins are mostly distinct
        if (hist && ci < total) atomicAdd(&hist[fixed_bin(kk, bkmin, bsh)], 1);
    }
}

// The same copy for two workgroups per CU, where the select's VALU work
// binds: keys at lds[i], words (list << kPosBits | token) at
// lds[kOffCand + i]. nzl lists the row's n_nz
// nonempty sub-chunks in position order, each as (index of its first
// candidate << kNzSubBits | sub-chunk). Thread t copies the N consecutive
// indices N t .. N t + N - 1: one binary search over nzl finds the entry of
// the first, and since every listed sub-chunk holds at least one candidate,
// index N t + u lies at most u entries further, which one batch of N reads
// settles. All loads are issued before any is used, so the copy costs one
// search chain and one memory round trip (indices past the end repeat the
// last candidate's load). Tracks this thread's min / max key.
// With fixed bins (hist != nullptr), every candidate is also counted in
// hist at bin min((key - bkmin) >> bsh, kHistBins - 1).
template <int N, int kOffCand>
__device__ __forceinline__ void copy_candidates_runs(const uint2* __restrict__ cand, const int* nzl,
                                                int n_nz, int total, uint32_t* lds,
                                                uint32_t& kmin, uint32_t& kmax, int* hist,
                                                uint32_t bkmin, int bsh) {
    const int tid = threadIdx.x;
    const int i0 = min(N * tid, total - 1);
    int k = 0;   // the last entry whose first index is <= i0
#pragma unroll
    for (int step = kSelMaxSub / 2; step > 0; step >>= 1) {
        const int t = k + step;
        if (t < n_nz && (nzl[min(t, n_nz - 1)] >> kNzSubBits) <= i0) k = t;
    }
    int ent[N];   // entries k .. k + N - 1 (the last one repeated past the list)
#pragma unroll
    for (int v = 0; v < N; ++v) ent[v] = nzl[min(k + v, n_nz - 1)];
    uint2 rec[N];
#pragma unroll
    for (int u = 0; u < N; ++u) {
        const int i = min(N * tid + u, total - 1);
        int e = ent[0];
#pragma unroll
        for (int v = 1; v <= u && v < N; ++v)
            if ((ent[v] >> kNzSubBits) <= i) e = ent[v];
        const int sc = e & ((1 << kNzSubBits) - 1);
        rec[u] = cand[static_cast<int64_t>(sc) * kSub + (i - (e >> kNzSubBits))];
    }
    uint32_t kk[N], cw[N];
#pragma unroll
    for (int u = 0; u < N; ++u) {
        kk[u] = float_key(__uint_as_float(rec[u].x));
        cw[u] = rec[u].y;
    }
    // the thread's N slots (< N * kSelThreads <= the LDS capacity; slots past
    // total are never read), 16 bytes per store when N allows
    if constexpr (N % 4 == 0) {
#pragma unroll
        for (int u = 0; u < N; u += 4) {
            *reinterpret_cast<uint4*>(lds + N * tid + u) = make_uint4(kk[u], kk[u + 1], kk[u + 2], kk[u + 3]);
            *reinterpret_cast<uint4*>(lds + kOffCand + N * tid + u) =
                make_uint4(cw[u], cw[u + 1], cw[u + 2], cw[u + 3]);
        }
    } else {
#pragma unroll
        for (int u = 0; u < N; ++u) {
            lds[N * tid + u] = kk[u];
            lds[kOffCand + N * tid + u] = cw[u];
        }
    }
#pragma unroll
    for (int u = 0; u < N; ++u) {
        if (N * tid + u < total) {
            kmin = min(kmin, kk[u]);
            kmax = max(kmax, kk[u]);
            // one LDS atomic per candidate: their bins are mostly distinct
            if (hist) atomicAdd(&hist[fixed_bin(kk[u], bkmin, bsh)], 1);
        }
    }
}

// Emit T as token ids in candidate order (each thread owns a contiguous
// range of candidate indices) and the per-list sums of exp(l~ - shift) over
// the unselected candidates (candidates are in list-major order, so a thread
// adds one partial per run of equal list ids).
// Variant Bx (Appendix B) in the top-k stage: the background value of list
// j is the mean of its unselected members, and its Eq. 4 term splits into
// W_j |R_j| v_bar_j minus W_j times the selected rows of the list, with
// W_j = M_j / |B n R_j|. The row forms W_j here, from the same masses as the
// background role (the scan's below-threshold segments of the list, scaled to
// the row's shift, plus its unselected candidates), and hands every entry of
// T its list's W_j. Thread t owns lists t + u * kSelThreads; their offsets are
// loaded when the row starts where one workgroup holds a CU (with two, the
// registers they would take cost the second workgroup its place), else with
// the masses.
constexpr int kBxPer = kMaxLists / kSelThreads;
static_assert(kMaxLists % kSelThreads == 0, "whole list strides");
struct BxRow {
    int lo[kBxPer], hi[kBxPer];   // the thread's lists in the list-major order (preloaded)
    const int32_t* loff;          // list starts of this head
    const float* segs;            // below-threshold masses of this head, stride G
    int seg_stride;
    float tlo;                    // the row's threshold tau_lo
    bool rescan;                  // the row took the re-scan path (no below-threshold masses)
    float* bx_w;                  // [n_list] W_j of the row
    float* bx_wsel;               // [max_topk] W of the list of each entry of T
};

template <bool kBx, bool kBxPre, typename KeyAt, typename CandAt, typename IsSel>
__device__ __forceinline__ void emit_selection(KeyAt key_at, CandAt cand_at, IsSel is_sel,
                                               int total, int k, int n_list,
                                               float shift, unsigned long long* mass,
                                               int32_t* sel_tok, float* cand_mass,
                                               const BxRow& bx, SelectScratch& ss) {
    const int tid = threadIdx.x;
    const int eper = (total + kSelThreads - 1) / kSelThreads;
    const int e0 = min(tid * eper, total);
    const int e1 = min(e0 + eper, total);
    int nsel = 0;
    for (int i = e0; i < e1; ++i) nsel += is_sel(i, key_at(i), cand_at(i)) ? 1 : 0;
    int tot = 0;
    int o = block_excl_scan<kSelThreads, false>(nsel, tot, ss);   // ss is not written before the barrier below
    const int o_first = o;
    int run_list = -1;
    unsigned long long run = 0ull;
    for (int i = e0; i < e1; ++i) {
        const uint32_t key = key_at(i);
        const uint32_t cand = cand_at(i);
        const int lst = static_cast<int>(cand >> kPosBits);
        if (lst != run_list) {
            if (run) atomicAdd(&mass[run_list], run);
            run = 0ull;
            run_list = lst;
        }
        if (is_sel(i, key, cand)) {
            if (o < k) sel_tok[o] = static_cast<int32_t>(cand & kPosMask);
            ++o;
        } else {
            run += static_cast<unsigned long long>(__expf(key_float(key) - shift) * kMassScale);
        }
    }
    if (run) atomicAdd(&mass[run_list], run);
    __syncthreads();
    if constexpr (!kBx) {
        for (int j = tid; j < n_list; j += kSelThreads)
            cand_mass[j] = static_cast<float>(mass[j]) * kMassUnscale;
    } else {
        const float neg_inf = -__builtin_huge_valf();
        const bool live = shift != neg_inf;
        const bool use_below = live && bx.tlo != neg_inf && !bx.rescan;
        const float below_scale = use_below ? __expf(bx.tlo - shift) : 0.0f;
        float mj[kBxPer];
        int sz[kBxPer];
#pragma unroll
        for (int u = 0; u < kBxPer; ++u) {
            const int j = tid + u * kSelThreads;
            mj[u] = 0.0f;
            sz[u] = 0;
            if (j < n_list) {
                const float cm = static_cast<float>(mass[j]) * kMassUnscale;
                cand_mass[j] = cm;
                float below = 0.0f;
                const int lo = kBxPre ? bx.lo[u] : bx.loff[j];
                const int hi = kBxPre ? bx.hi[u] : bx.loff[j + 1];
                sz[u] = hi - lo;
                if (use_below && hi > lo)
                    for (int sg = j + lo / kSub; sg <= j + (hi - 1) / kSub; ++sg)
                        below += bx.segs[sg * bx.seg_stride];
                mj[u] = live ? below * below_scale + cm : 0.0f;
            }
        }
        // the masses are read: their words now hold |T n R_j| and then W_j
        __syncthreads();
        int* cnt = reinterpret_cast<int*>(mass);
        float* wl = reinterpret_cast<float*>(mass) + n_list;
        for (int j = tid; j < n_list; j += kSelThreads) cnt[j] = 0;
        __syncthreads();
        o = o_first;
        for (int i = e0; i < e1; ++i) {
            const uint32_t cand = cand_at(i);
            if (is_sel(i, key_at(i), cand)) {
                if (o < k) atomicAdd(&cnt[cand >> kPosBits], 1);
                ++o;
            }
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kBxPer; ++u) {
            const int j = tid + u * kSelThreads;
            if (j < n_list) {
                const int un = sz[u] - cnt[j];
                const float W = un > 0 ? mj[u] / static_cast<float>(un) : 0.0f;
                wl[j] = W;
                bx.bx_w[j] = W;
            }
        }
        __syncthreads();
        o = o_first;
        for (int i = e0; i < e1; ++i) {
            const uint32_t cand = cand_at(i);
            if (is_sel(i, key_at(i), cand)) {
                if (o < k) bx.bx_wsel[o] = wl[cand >> kPosBits];
                ++o;
            }
        }
    }
}

// Score every indexed token of a row again from its head's LUT (the re-scan
// path): keys and words into comp_key / comp_pos in position order.
template <typename PQ>
__device__ __forceinline__ void rescan_row(const Dims& D, const Index& ix, const Work& w,
                                           float* lut_s, int bg, int hh, int n_r, int64_t base,
                                           int64_t rbase) {
    stage_head_lut<PQ, kSelThreads>(lut_s, w.lut + static_cast<int64_t>(bg) * PQ::LUT_ROW * D.G,
                                    D.G, hh);
    __syncthreads();
    const typename PQ::Code* codes = reinterpret_cast<const typename PQ::Code*>(ix.codes) + base;
    const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * D.G;
    for (int pos = threadIdx.x; pos < n_r; pos += kSelThreads) {
        const uint32_t wd = ix.pos_word[base + pos];
        const int j = static_cast<int>(wd >> kPosBits);
        float fs[1];
        fine_sum<PQ, 1>(lut_s, codes[pos], fs);
        const float sc = pq_logit(ix.norms[base + pos], coarse[j * D.G + hh], fs[0]);
        w.comp_key[rbase + pos] = float_key(sc);
        w.comp_pos[rbase + pos] = static_cast<int32_t>(wd);
    }
}

template <bool kDev, int kCap, bool kBx>
__device__ __forceinline__ void select_row(const Dims& D, const BatchArgs& ba, const Index& ix,
                                           const Work& w, int force_fallback) {
    using L = SelLayout<kCap>;
    constexpr int kOffCand = L::kOffCand;
    extern __shared__ uint32_t lds[];
    unsigned long long* mass = reinterpret_cast<unsigned long long*>(lds + L::kOffMass);
    int* hist = reinterpret_cast<int*>(lds + L::kOffHist);
    uint32_t* r_key = lds + L::kOffRKey;
    int* r_idx = reinterpret_cast<int*>(lds + L::kOffRIdx);
    int* r_tok = reinterpret_cast<int*>(lds + L::kOffRTok);
    uint32_t* chosen = lds + L::kOffBits;
    int* counter = reinterpret_cast<int*>(lds + L::kOffCounter);
    // the copy by nonempty sub-chunks where two workgroups share a CU (1.2 us
    // faster at 512 rows), by a search of every index over the sub-chunk
    // offsets with one workgroup per CU (0.4 us faster at 32 rows: its loads
    // of neighbouring lanes touch neighbouring slots)
    constexpr bool kRunsCopy = kCap == kSelCapSmall;
    int* subl = reinterpret_cast<int*>(lds + L::kOffSub);
    __shared__ SelectScratch ss;
    __shared__ BlockScratch bs;
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wave = tid / kWave;
    const int row = blockIdx.x;
    const int b = row / D.Hq;
    const int h = row % D.Hq;
    const int g = h / D.G;
    const int hh = h % D.G;
    const int bg = b * D.Hkv + g;
    const int n_r = arg_n_r<kDev>(ba, w, b);
    const int k = arg_topk<kDev>(ba, w, b);
    const int nsub = (n_r + kSub - 1) / kSub;
    const int64_t rbase = static_cast<int64_t>(row) * D.rcap;
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    int32_t* sel_tok = w.sel_tok + static_cast<int64_t>(row) * D.max_topk;
    float* cand_mass = w.cand_mass + static_cast<int64_t>(row) * D.n_list;
    const float neg_inf = -__builtin_huge_valf();

    for (int j = tid; j < D.n_list; j += kSelThreads) mass[j] = 0ull;
    for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = 0;
    for (int i = tid; i < kCap / 32; i += kSelThreads) chosen[i] = 0u;
    if (tid < 4) counter[tid] = 0;   // counter[1] is the equal-key flag of the rank
    BxRow bx{};
    constexpr bool kBxPre = kCap != kSelCapSmall;
    if constexpr (kBx) {
        bx.loff = ix.loff + static_cast<int64_t>(bg) * (D.n_list + 1);
        if constexpr (kBxPre) {
#pragma unroll
            for (int u = 0; u < kBxPer; ++u) {
                const int j = tid + u * kSelThreads;
                bx.lo[u] = j < D.n_list ? bx.loff[j] : 0;
                bx.hi[u] = j < D.n_list ? bx.loff[j + 1] : 0;
            }
        }
        bx.segs = w.seg_sum + static_cast<int64_t>(bg) * D.nseg_cap * D.G + hh;
        bx.seg_stride = D.G;
        bx.tlo = w.tau_lo[row];
        bx.bx_w = w.bx_w + static_cast<int64_t>(row) * D.n_list;
        bx.bx_wsel = w.bx_wsel + static_cast<int64_t>(row) * D.max_topk;
    }

    // 1) candidate counts: wave w owns sub-chunks [w * spw, (w + 1) * spw)
    const bool small_nsub = nsub <= kSelMaxSub;
    const int spw = small_nsub ? (nsub + kNW - 1) / kNW : 0;
    const int32_t* cnt = w.cand_cnt + static_cast<int64_t>(row) * D.nsub_cap;
    int c_l = 0, incl = 0;
    int total = 0;
    int n_nz = 0;   // nonempty sub-chunks of the row
    if (small_nsub) {
        const int sc = wave * spw + lane;
        c_l = (lane < spw && sc < nsub) ? cnt[sc] : 0;
        incl = wave_incl_scan_i32(c_l);
        const uint64_t nzm = kRunsCopy ? __builtin_amdgcn_ballot_w64(c_l > 0) : 0ull;
        if (lane == kWave - 1) {
            ss.wave_tot[wave] = incl;
            ss.wave_aux[wave] = __popcll(nzm);
        }
        __syncthreads();
        int wbase = 0, nzbase = 0;
#pragma unroll
        for (int i = 0; i < kNW; ++i) {
            const int t = ss.wave_tot[i];
            const int z = ss.wave_aux[i];
            wbase += i < wave ? t : 0;
            nzbase += i < wave ? z : 0;
            total += t;
            n_nz += z;
        }
        incl += wbase;   // row-wide inclusive offset of this lane's sub-chunk
        if constexpr (kRunsCopy) {
            if (c_l > 0) subl[nzbase + lanes_below(nzm)] = ((incl - c_l) << kNzSubBits) | sc;
        } else {
            if (lane < spw && sc < nsub) subl[sc] = incl - c_l;
        }
        __syncthreads();
    } else {
        int mine = 0;
        const int per = (nsub + kSelThreads - 1) / kSelThreads;
        const int sc0 = min(tid * per, nsub), sc1 = min(sc0 + per, nsub);
        for (int sc = sc0; sc < sc1; ++sc) mine += cnt[sc];
        block_excl_scan<kSelThreads>(mine, total, ss);
    }
    const bool fallback = force_fallback || (n_r > 0 && total < (k > 0 ? k : 1));
    bx.rescan = fallback;
    float shift = neg_inf;

    if (!fallback && small_nsub && total <= kCap) {
        // ---- fast path: candidates in LDS, position order ----
        auto KEY = [&](int i) { return lds[i]; };
        auto CAND = [&](int i) { return lds[kOffCand + i]; };
        uint32_t kmin = 0xffffffffu, kmax = 0u, kcount = 0u;
        const uint2* cand = w.cand + rbase;
        // Bins fixed in advance from the sampled range [tau_lo, tau_hi] (every
        // candidate is >= tau_lo; those above tau_hi share the last bin), so
        // the histogram is built during the copy; otherwise from the
        // candidates' own min / max in a second pass.
        const float tlo = w.tau_lo[row], thi = w.tau_hi[row];
        const bool fixed = k > 0 && tlo > neg_inf && thi > tlo && thi < -neg_inf;
        uint32_t bkmin = fixed ? float_key(tlo) : 0u;
        int bsh = fixed ? bin_shift(bkmin, float_key(thi)) : 0;
        int* fh = fixed ? hist : nullptr;
        constexpr int kMid = kCap / kSelThreads > 8 ? 8 : kCap / kSelThreads;
        auto copy = [&](auto tier) {
            constexpr int N = decltype(tier)::value;
            if constexpr (kRunsCopy)
                copy_candidates_runs<N, kOffCand>(cand, subl, n_nz, total, lds, kmin, kmax, fh, bkmin, bsh);
            else
                copy_candidates_search<N, kOffCand>(cand, subl, nsub, total, lds, kmin, kmax, fh, bkmin, bsh);
        };
        if (total > kMid * kSelThreads)
            copy(std::integral_constant<int, kCap / kSelThreads>{});
        else if (total > 4 * kSelThreads)
            copy(std::integral_constant<int, kMid>{});
        else if (total > 0)
            copy(std::integral_constant<int, 4>{});
        if (!fixed) block_min_max_count<kSelThreads>(kmin, kmax, kcount, bs);
        auto TOK = [&](int i) { return static_cast<int>(CAND(i) & kPosMask); };
        if (k == 0) {
            shift = total > 0 ? key_float(kmax) : neg_inf;
            emit_selection<kBx, kBxPre>(
                KEY, CAND, [](int, uint32_t, uint32_t) { return false; }, total, 0, D.n_list, shift,
                mass, sel_tok, cand_mass, bx, ss);
        } else {
            if (!fixed) {
                bkmin = kmin;
                bsh = bin_shift(kmin, kmax);
                for (int i0 = 0; i0 < total; i0 += kSelThreads) {
                    const int i = i0 + tid;
                    const bool act = i < total;
                    if (act) atomicAdd(&hist[fixed_bin(KEY(i), bkmin, bsh)], 1);
                }
            }
            __syncthreads();
            // one wave finds the boundary bin and broadcasts it
            if (tid < kWave) {
                int ab = 0;
                const int bin = wave_find_bin_desc(hist, k, ab);
                if (tid == 0) {
                    bs.bcast[0] = bin;
                    bs.bcast[1] = ab;
                }
            }
            __syncthreads();
            const int bstar = bs.bcast[0];
            const int above = bs.bcast[1];
            uint32_t kth = 0u;
            const bool by_rank = rank_boundary_bin(KEY, TOK, total, bkmin, bsh, bstar, hist[bstar],
                                                   k - above, r_key, r_idx, r_tok, counter,
                                                   counter + 1, chosen, kth, bs);
            if (by_rank) {
                shift = key_float(kth);   // the k-th largest score
                emit_selection<kBx, kBxPre>(
                    KEY, CAND,
                    [&](int i, uint32_t key, uint32_t) {
                        const int bn = static_cast<int>(fixed_bin(key, bkmin, bsh));
                        return bn > bstar || (bn == bstar && ((chosen[i >> 5] >> (i & 31)) & 1u));
                    },
                    total, k, D.n_list, shift, mass, sel_tok, cand_mass, bx, ss);
            } else {
                // very dense boundary bin: radix select
                const SelectResult r = block_select_desc<kSelThreads>(
                    KEY, [](int) { return true; }, total, k, ss);
                const uint32_t kk = r.key;
                const int need_r = k - r.count_above;
                int tok_cut = 0x7fffffff;
                if (r.count_equal > need_r) {
                    const SelectResult t = block_select_desc<kSelThreads>(
                        [&](int i) { return ~static_cast<uint32_t>(TOK(i)); },
                        [&](int i) { return KEY(i) == kk; }, total, need_r, ss);
                    tok_cut = static_cast<int>(~t.key);
                }
                shift = key_float(kk);
                emit_selection<kBx, kBxPre>(
                    KEY, CAND,
                    [&](int, uint32_t key, uint32_t cw) {
                        return key > kk || (key == kk && static_cast<int>(cw & kPosMask) <= tok_cut);
                    },
                    total, k, D.n_list, shift, mass, sel_tok, cand_mass, bx, ss);
            }
        }
    } else {
        // ---- slow path: candidates in global memory (many, or the re-scan) ----
        if (!fallback) {
            const int per = (nsub + kSelThreads - 1) / kSelThreads;
            const int sc0 = min(tid * per, nsub), sc1 = min(sc0 + per, nsub);
            int mine = 0;
            for (int sc = sc0; sc < sc1; ++sc) mine += cnt[sc];
            int tot = 0;
            int o = block_excl_scan<kSelThreads>(mine, tot, ss);
            for (int sc = sc0; sc < sc1; ++sc) {
                const int c = cnt[sc];
                const int64_t src = rbase + static_cast<int64_t>(sc) * kSub;
                for (int i = 0; i < c; ++i, ++o) {
                    const uint2 rec = w.cand[src + i];
                    w.comp_key[rbase + o] = float_key(__uint_as_float(rec.x));
                    w.comp_pos[rbase + o] = static_cast<int32_t>(rec.y);
                }
            }
        } else {
            float* lut_s = reinterpret_cast<float*>(lds);   // at most 16 KB of the key area
            if (D.pq_bits == 4)
                rescan_row<Pq4>(D, ix, w, lut_s, bg, hh, n_r, base, rbase);
            else
                rescan_row<Pq8>(D, ix, w, lut_s, bg, hh, n_r, base, rbase);
            total = n_r;
        }
        __syncthreads();
        const uint32_t* ckey = w.comp_key + rbase;
        const uint32_t* ccand = reinterpret_cast<const uint32_t*>(w.comp_pos + rbase);
        auto KEY = [&](int i) { return ckey[i]; };
        auto CAND = [&](int i) { return ccand[i]; };
        if (total == 0) {
            shift = neg_inf;
            emit_selection<kBx, kBxPre>(KEY, CAND, [](int, uint32_t, uint32_t) { return false; }, 0, 0,
                           D.n_list, shift, mass, sel_tok, cand_mass, bx, ss);
        } else {
            const SelectResult r = block_select_desc<kSelThreads>(
                KEY, [](int) { return true; }, total, k > 0 ? k : 1, ss);
            const uint32_t kth = k > 0 ? r.key : 0xffffffffu;
            int tok_cut = 0x7fffffff;
            if (k > 0 && r.count_equal > k - r.count_above) {
                const SelectResult t = block_select_desc<kSelThreads>(
                    [&](int i) { return ~(ccand[i] & kPosMask); },
                    [&](int i) { return ckey[i] == kth; }, total, k - r.count_above, ss);
                tok_cut = static_cast<int>(~t.key);
            }
            shift = key_float(r.key);   // k-th largest, or the maximum when k = 0
            emit_selection<kBx, kBxPre>(
                KEY, CAND,
                [&](int, uint32_t key, uint32_t cand) {
                    return k > 0 && (key > kth || (key == kth && static_cast<int>(cand & kPosMask) <= tok_cut));
                },
                total, k, D.n_list, shift, mass, sel_tok, cand_mass, bx, ss);
        }
    }
    if (tid == 0) {
        w.row_shift[row] = shift;
        w.row_flag[row] = fallback ? 1 : 0;
    }
}

template <bool kDev, bool kBx>
__global__ __launch_bounds__(kSelThreads) void select_kernel(Dims D, BatchArgs ba, Index ix, Work w,
                                                             int force_fallback) {
    select_row<kDev, kSelCap, kBx>(D, ba, ix, w, force_fallback);
}

// Two of these share a CU only when each wave holds at most 80 SGPRs (the
// few beyond that spill to VGPR lanes).
template <bool kDev, bool kBx>
__global__ __launch_bounds__(kSelThreads) __attribute__((amdgpu_num_sgpr(80))) void select_small_kernel(
    Dims D, BatchArgs ba, Index ix, Work w, int force_fallback) {
    select_row<kDev, kSelCapSmall, kBx>(D, ba, ix, w, force_fallback);
}

// The small-capacity select when the rows outnumber the CUs and two of its
// workgroups fit in one CU's LDS.
static bool select_small(const Dims& D) {
    const int n_cu = device_cu_count();
    constexpr size_t kLdsPerCu = 160 * 1024;
    constexpr size_t kStatic = sizeof(SelectScratch) + sizeof(BlockScratch);
    return n_cu > 0 && D.B * D.Hq > n_cu &&
           2 * (SelLayout<kSelCapSmall>::bytes(D.n_list) + kStatic) <= kLdsPerCu;
}

template <bool kDev, bool kBx>
static void launch_select_d(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                            int force_fallback, hipStream_t s, const KTiming& tm) {
    if (select_small(D))
        hipExtLaunchKernelGGL((select_small_kernel<kDev, kBx>), dim3(D.B * D.Hq), dim3(kSelThreads),
                              SelLayout<kSelCapSmall>::bytes(D.n_list), s, tm.start, tm.stop, 0, D, ba,
                              ix, w, force_fallback);
    else
        hipExtLaunchKernelGGL((select_kernel<kDev, kBx>), dim3(D.B * D.Hq), dim3(kSelThreads),
                              SelLayout<kSelCap>::bytes(D.n_list), s, tm.start, tm.stop, 0, D, ba, ix,
                              w, force_fallback);
}

hipError_t launch_select(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                         int force_fallback, bool bx, hipStream_t s, const KTiming& tm) {
    if (w.ba_dev && bx)
        launch_select_d<true, true>(D, ba, ix, w, force_fallback, s, tm);
    else if (w.ba_dev)
        launch_select_d<true, false>(D, ba, ix, w, force_fallback, s, tm);
    else if (bx)
        launch_select_d<false, true>(D, ba, ix, w, force_fallback, s, tm);
    else
        launch_select_d<false, false>(D, ba, ix, w, force_fallback, s, tm);
    return hipGetLastError();
}

hipError_t configure_select() {
    const void* k[] = {reinterpret_cast<const void*>(&select_kernel<false, false>),
                       reinterpret_cast<const void*>(&select_kernel<true, false>),
                       reinterpret_cast<const void*>(&select_kernel<false, true>),
                       reinterpret_cast<const void*>(&select_kernel<true, true>),
                       reinterpret_cast<const void*>(&select_small_kernel<false, false>),
                       reinterpret_cast<const void*>(&select_small_kernel<true, false>),
                       reinterpret_cast<const void*>(&select_small_kernel<false, true>),
                       reinterpret_cast<const void*>(&select_small_kernel<true, true>)};
    const int big = static_cast<int>(SelLayout<kSelCap>::bytes(kMaxLists));
    const int small = static_cast<int>(SelLayout<kSelCapSmall>::bytes(kMaxLists));
    const int bytes[] = {big, big, big, big, small, small, small, small};
    hipError_t e = hipSuccess;
    for (int i = 0; i < 8 && e == hipSuccess; ++i)
        e = hipFuncSetAttribute(k[i], hipFuncAttributeMaxDynamicSharedMemorySize, bytes[i]);
    return e;
}

}  // namespace pqhsa
