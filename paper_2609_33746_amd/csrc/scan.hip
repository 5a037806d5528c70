// Code scan (Section 3.1, Eq. 2; Section 3.3, execution path: the scan and
// the per-list reduction of the background run in one pass). Every indexed
// token of every list is scored for the G query heads that share its KV
// head, in one pass over the list-major codes.
//
// Work decomposition: the list-major positions of each (batch element, KV
// head) are cut into sub-chunks of kSub positions; one wave owns one
// sub-chunk, and a workgroup holds kScanWaves consecutive sub-chunks (a
// chunk) of the same KV head so that they share one copy of the group LUT in
// LDS; when the grid would take several rounds of the device, a workgroup
// scans up to four chunks of its KV head with one staging of its tables. Every
// batch element gets the workgroup count of the longest R_b; the surplus
// workgroups of shorter sequences exit at once. The workgroups of one KV head
// are spaced by the number of (batch element, KV head) units in the grid, so
// that they share an XCD.
//
// The workgroup first stages the group LUT in LDS (through registers), then
// each wave issues the loads of all its 64-position steps (list ids, codes,
// norms) at once, in step order, so the arithmetic of the first steps
// overlaps the arrival of the later ones; each lane gathers the coarse terms
// of its list from the group's coarse table.
//
// Per token and head the wave computes l~ and then either
//   * emits (l~, list id and token id) as a top-k candidate when
//     l~ >= tau_lo (the sampled threshold of its row), compacted in position
//     order at the start of the sub-chunk's own region of the row's candidate
//     buffer, or
//   * adds exp(l~ - tau_lo) (< 1) to the running mass of its inverted list.
// Tokens below tau_lo can never be in the top-k (tau_lo <= the k-th largest
// score whenever at least k candidates exist), so these masses are exactly
// the "below threshold" part of M_j in Eq. 4; the unselected candidates are
// added by the top-k stage.
//
// Masses are stored per (list j, sub-chunk s) pair at segment j + s of the KV
// head's segment array: along the list-major order neither j nor s decreases
// and each new pair increases at least one of them, so distinct pairs get
// distinct segments (some segment indices stay unused). No atomics are used
// and the result does not depend on scheduling.
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "pq_score.h"
#include "pqhsa_internal.h"

namespace pqhsa {

constexpr int kScanThreads = kScanWaves * kWave;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kIters = kSub / kWave;   // 64-position steps per sub-chunk
// The G coarse terms of one list, [n_list][G] layout.
template <int G>
__device__ __forceinline__ void load_coarse(const float* p, float (&v)[G]) {
    if constexpr (G == 8) {
        const float4 a = reinterpret_cast<const float4*>(p)[0];
        const float4 c = reinterpret_cast<const float4*>(p)[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = c.x; v[5] = c.y; v[6] = c.z; v[7] = c.w;
    } else if constexpr (G == 4) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    } else if constexpr (G == 2) {
        const float2 a = *reinterpret_cast<const float2*>(p);
        v[0] = a.x; v[1] = a.y;
    } else {
        v[0] = *p;
    }
}

// Store the wave's masses of one list segment and clear them.
template <int G>
__device__ __forceinline__ void flush_segment(float* seg_row, float (&acc)[G]) {
    float mine = 0.0f;
    if constexpr (G == 4) {
        // the four heads reduced together: two exchanges within each quad
        // leave lane l with its quad's sum of head l & 3, two row rotations
        // by 4 and 8 lanes sum the row's quads, and two lane swaps between
        // rows (16 and 32 apart) sum the rows
        const int lane = lane_id();
        const bool b0 = lane & 1, b1 = lane & 2;
        const float p = (b0 ? acc[1] : acc[0]) + dpp<0xB1>(b0 ? acc[0] : acc[1]);   // quad_perm [1,0,3,2]
        const float q = (b0 ? acc[3] : acc[2]) + dpp<0xB1>(b0 ? acc[2] : acc[3]);
        float u = (b1 ? q : p) + dpp<0x4E>(b1 ? p : q);                            // quad_perm [2,3,0,1]
        u += dpp<0x124>(u);   // row_ror:4
        u += dpp<0x128>(u);   // row_ror:8
        const uint32_t ub = __float_as_uint(u);
        const auto r16 = __builtin_amdgcn_permlane16_swap(ub, ub, false, false);
        u = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
        const uint32_t vb = __float_as_uint(u);
        const auto r32 = __builtin_amdgcn_permlane32_swap(vb, vb, false, false);
        mine = __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
#pragma unroll
        for (int hh = 0; hh < G; ++hh) acc[hh] = -0.0f;
    } else {
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            const float tot = wave_sum(acc[hh]);
            if (lane_id() == hh) mine = tot;
            acc[hh] = -0.0f;
        }
    }
    if (lane_id() < G) seg_row[lane_id()] = mine;
}

// Floats of the group LUT as staged in LDS: Pq8 [M][K][G]; Pq4 replicated
// (kRep4 interleaved copies, conflict-free lookups).
template <typename PQ, int G>
constexpr int kScanLutFloats = std::is_same<PQ, Pq4>::value ? kRep4Floats : PQ::LUT_ROW * G;

// G = heads scored per workgroup; GT = heads of the KV head's group (the
// stride of the group tables, masses and rows). A group of GT = 8 heads is
// split over two workgroups of G = 4: their tables then take 80 KB of LDS,
// so two workgroups share a CU instead of one (the codes are read twice).
// At most 80 SGPRs per wave (a few spill to VGPR lanes): with more, a second
// workgroup does not fit on the CU.
template <int G, int GT, typename PQ, bool kDev>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_num_sgpr(80))) void scan_kernel(
    Dims D, BatchArgs ba, Index ix, Work w, int nwg, int nwg_grid) {
    // the group LUT at a compile-time LDS address (so that an entry address
    // is one shift of a code)
    __shared__ float4 lut4[kScanLutFloats<PQ, G> / 4];
    float* lut_s = reinterpret_cast<float*>(lut4);
    constexpr int kParts = GT / G;   // workgroups per (b, g) and sub-chunk range
    static_assert(kParts * G == GT, "head split");
    // workgroup i serves unit i mod U of the U = B Hkv kParts (b, g, part)
    // units, chunks c, c + nwg_grid, c + 2 nwg_grid, ... (c = i / U) of the
    // unit's nwg chunks, with the tables staged once: workgroups run on XCD
    // i mod 8, so when U is a multiple of 8 every workgroup of a unit shares
    // one XCD and its L2, and the unit's tables come from HBM once instead of
    // once per XCD
    const int n_units = D.B * D.Hkv * kParts;
    const int unit = blockIdx.x % n_units;
    const int part = unit % kParts;
    const int bg = unit / kParts;
    const int b = bg / D.Hkv;
    const int g = bg % D.Hkv;
    const int n_r = arg_n_r<kDev>(ba, w, b);
    const int chunk0 = blockIdx.x / n_units;
    if (chunk0 * kScanWaves * kSub >= n_r) return;   // surplus workgroup of a shorter sequence

    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = lane_id();
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const int row0 = b * D.Hq + g * GT + part * G;
    // this workgroup's G heads within the group tables ([..][GT] layouts)
    const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * GT + part * G;

    // 1) the tables shared by the workgroup, and the thresholds
    constexpr int kStage = kScanLutFloats<PQ, G> / 4 / kScanThreads;
    static_assert(kStage * kScanThreads * 4 == kScanLutFloats<PQ, G>, "LUT staging tiling");
    const float* glut = w.lut + static_cast<int64_t>(bg) * PQ::LUT_ROW * GT + part * G;
    float4 st[kStage];
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
        const int f4 = i * kScanThreads + tid;
        if constexpr (std::is_same<PQ, Pq4>::value) {
            // float t of replicated row `entry` is component (f mod G) of the entry
            const int entry = f4 / 16;
            const int f = (f4 % 16) * 4;
            const float* src = glut + entry * GT;
            st[i] = make_float4(src[f % G], src[(f + 1) % G], src[(f + 2) % G], src[(f + 3) % G]);
        } else if constexpr (G == GT) {
            st[i] = reinterpret_cast<const float4*>(glut)[f4];
        } else {
            // float4 f4 of the [M][K][G] slice: entry f4 * 4 / G, heads from (f4 * 4) mod G
            const int f = f4 * 4;
            st[i] = *reinterpret_cast<const float4*>(glut + (f / G) * GT + f % G);
        }
    }
    float tlo[G], tlo_l2e[G];   // tau_lo, and tau_lo log2(e) for the masses' exp2
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        tlo[hh] = w.tau_lo[row0 + hh];
        tlo_l2e[hh] = tlo[hh] * kLog2e;
    }
    float4* ldst = reinterpret_cast<float4*>(lut_s);
#pragma unroll
    for (int i = 0; i < kStage; ++i) ldst[i * kScanThreads + tid] = st[i];
    __syncthreads();
    for (int chunk = chunk0; chunk < nwg; chunk += nwg_grid) {
        const int sc = chunk * kScanWaves + wave;
        const int p_begin = sc * kSub;
        const int p_end = min(p_begin + kSub, n_r);
        if (p_begin >= n_r) break;   // later chunks start later still
        // 2) per 64-position step: list ids, codes and norms (addresses clamped
        //    into R_b, so every load is in bounds), issued in the order the steps
        //    use them, after the tables: each step waits only for its own data
        const typename PQ::Code* codes = reinterpret_cast<const typename PQ::Code*>(ix.codes) + base;
        uint32_t wl[kIters];   // list id << kPosBits | token id
        typename PQ::Code cv[kIters];
        float rv[kIters];
#pragma unroll
        for (int it = 0; it < kIters; ++it) {
            const int p = min(p_begin + it * kWave + lane, n_r - 1);
            wl[it] = ix.pos_word[base + p];
            cv[it] = codes[p];
            rv[it] = ix.norms[base + p];
        }
        float* segs = w.seg_sum + (static_cast<int64_t>(bg) * D.nseg_cap + sc) * GT + part * G;   // + j * GT
        int cur = __builtin_amdgcn_readfirstlane(static_cast<int>(wl[0] >> kPosBits));   // open segment's list
        float acc[G];
        int cbase[G];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) { acc[hh] = -0.0f; cbase[hh] = 0; }   // -0 + x folds to x

#pragma unroll
        for (int it = 0; it < kIters; ++it) {
            const int p_first = p_begin + it * kWave;
            if (p_first >= p_end) continue;   // uniform: past the end of a short last sub-chunk
            const int p = p_first + lane;
            const bool valid = p < p_end;
            const uint64_t vmask = __builtin_amdgcn_ballot_w64(valid);
            // coarse terms of the lanes' lists, gathered from the group table
            // (neighbouring lanes mostly share a list; staging the table in
            // LDS instead was a little slower, 12.4 against 12.3 us at 128K
            // and 97.4 against 96.2 us at 16 sequences)
            const int j = static_cast<int>(wl[it] >> kPosBits);
            float cf[G];
            load_coarse<G>(coarse + j * GT, cf);
            float fs[G];
            if constexpr (std::is_same<PQ, Pq4>::value) fine_sum_rep4<G>(lut_s, cv[it], fs);
            else fine_sum<PQ, G>(lut_s, cv[it], fs);
            // exp(l~ - tau_lo) as exp2(r log2(e) (coarse + fine) - tau_lo log2(e)):
            // one FMA per head, with r log2(e) shared by the G heads
            const float r_l2e = rv[it] * kLog2e;
            float s[G], e[G];
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                const float x = cf[hh] + fs[hh];
                s[hh] = pq_logit(rv[it], cf[hh], fs[hh]);
                e[hh] = (valid && s[hh] < tlo[hh])
                            ? __builtin_amdgcn_exp2f(__builtin_fmaf(r_l2e, x, -tlo_l2e[hh]))
                            : 0.0f;
            }
            // close the lists that end inside this step (lists are contiguous and
            // ascending along the lanes)
            const int j_last = __builtin_amdgcn_readlane(j, min(p_end - p_first, kWave) - 1);
            while (cur != j_last) {
                const bool in = valid && j == cur;
#pragma unroll
                for (int hh = 0; hh < G; ++hh) acc[hh] += in ? e[hh] : 0.0f;
                flush_segment<G>(segs + cur * GT, acc);
                const int nxt = __popcll(__builtin_amdgcn_ballot_w64(j <= cur) & vmask);
                cur = __builtin_amdgcn_readlane(j, nxt);
            }
            {
                const bool in = valid && j == cur;
#pragma unroll
                for (int hh = 0; hh < G; ++hh) acc[hh] += in ? e[hh] : 0.0f;
            }
            // candidates >= tau_lo, compacted in position order
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                // ballots of bare compares, masked by the valid lanes' ballot,
                // stay lane masks in scalar registers
                const uint64_t mask = __builtin_amdgcn_ballot_w64(s[hh] >= tlo[hh]) & vmask;
                if (mask) {
                    if (valid && s[hh] >= tlo[hh]) {
                        const int64_t o = static_cast<int64_t>(row0 + hh) * D.rcap + p_begin +
                                          cbase[hh] + lanes_below(mask);
                        w.cand[o] = make_uint2(__float_as_uint(s[hh]), wl[it]);
                    }
                    cbase[hh] += __popcll(mask);
                }
            }
        }
        flush_segment<G>(segs + cur * GT, acc);
        int mine = 0;
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
            if (lane == hh) mine = cbase[hh];
        if (lane < G) w.cand_cnt[static_cast<int64_t>(row0 + lane) * D.nsub_cap + sc] = mine;
    }
}

constexpr size_t kScanLdsMax = 160 * 1024;   // LDS of one workgroup on gfx950
constexpr int kScanMaxChunks = 4;

template <int G, int GT, typename PQ, bool kDev>
static hipError_t launch_scan_d(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                                int nwg, hipStream_t s, const KTiming& tm) {
    static_assert(kScanLutFloats<PQ, G> * 4 <= kScanLdsMax, "LDS budget");
    const int n_units = D.B * D.Hkv * (GT / G);
    // chunks per workgroup: as many as the grid has rounds of the workgroups
    // that run at once (two per CU), at most kScanMaxChunks, each workgroup
    // staging its tables once for all of them (at 4 and 16 sequences 4
    // chunks per workgroup beat 1, 2, 8 and 16)
    const int n_cu = device_cu_count();
    const int64_t resident = static_cast<int64_t>(2) * (n_cu > 0 ? n_cu : 1);
    const int cpw = static_cast<int>(
        std::min<int64_t>(kScanMaxChunks, std::max<int64_t>(1, static_cast<int64_t>(n_units) * nwg / resident)));
    const int nwg_grid = (nwg + cpw - 1) / cpw;
    const dim3 grid(n_units * nwg_grid);
    hipExtLaunchKernelGGL((scan_kernel<G, GT, PQ, kDev>), grid, dim3(kScanThreads), 0, s, tm.start,
                          tm.stop, 0, D, ba, ix, w, nwg, nwg_grid);
    return hipGetLastError();
}

template <int G, int GT, typename PQ>
static hipError_t launch_scan_t(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                                int nwg, hipStream_t s, const KTiming& tm) {
    return w.ba_dev ? launch_scan_d<G, GT, PQ, true>(D, ba, ix, w, nwg, s, tm)
                    : launch_scan_d<G, GT, PQ, false>(D, ba, ix, w, nwg, s, tm);
}

template <typename PQ>
static hipError_t launch_scan_pq(const Dims& D, const BatchArgs& ba, const Index& ix,
                                 const Work& w, int nwg, hipStream_t s, const KTiming& tm) {
    switch (D.G) {
        case 1: return launch_scan_t<1, 1, PQ>(D, ba, ix, w, nwg, s, tm);
        case 2: return launch_scan_t<2, 2, PQ>(D, ba, ix, w, nwg, s, tm);
        case 4: return launch_scan_t<4, 4, PQ>(D, ba, ix, w, nwg, s, tm);
        case 8: return launch_scan_t<4, 8, PQ>(D, ba, ix, w, nwg, s, tm);   // two workgroups of 4 heads
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_scan(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w, int nwg,
                       hipStream_t s, const KTiming& tm) {
    if (nwg == 0) return hipSuccess;
    return D.pq_bits == 4 ? launch_scan_pq<Pq4>(D, ba, ix, w, nwg, s, tm)
                          : launch_scan_pq<Pq8>(D, ba, ix, w, nwg, s, tm);
}

}  // namespace pqhsa
