// Top-k selection (Section 3.2, Eq. 3): T = the k indexed tokens with the
// largest approximate logits, per (batch element, query head) row, ties to the
// smaller token id.
//
// Two kernels:
//  * sample_kernel (before the scan): scores a strided, list-stratified sample
//    of the row's list-major positions and takes a sample order statistic as
//    the candidate threshold tau_lo, chosen so that about twice k tokens of
//    the full row score at or above it.
//  * select_kernel (after the scan): gathers the candidates of the row (in
//    list-major position order), finds the exact k-th largest score by radix
//    select over order-preserving keys, breaks ties on token id with a second
//    radix select, writes T, and adds the unselected candidates to the
//    per-list background masses. If the threshold left fewer than k
//    candidates (or none at all), the row is re-scanned in full from the LUT
//    and every indexed token becomes a candidate; the below-threshold masses
//    of the scan are then ignored for that row. The result is exact either
//    way; only the cost differs.
#include "device_common.h"
#include "pq_score.h"
#include "pqhsa_internal.h"
#include "radix_select.h"

namespace pqhsa {

__device__ __forceinline__ int sample_stride(int n_r) {
    const int need = (n_r + kMaxSamples - 1) / kMaxSamples;
    return need > kSampleStride ? need : kSampleStride;
}

__global__ __launch_bounds__(kSelThreads) void sample_kernel(Dims D, BatchInts tk, Index ix,
                                                             Work w, float bias) {
    __shared__ float lut_s[kLutRow];
    __shared__ uint32_t keys[kMaxSamples];
    __shared__ SelectScratch sh;
    const int row = blockIdx.x;
    const int b = row / D.Hq;
    const int h = row % D.Hq;
    const int g = h / D.G;
    const int hh = h % D.G;
    const int bg = b * D.Hkv + g;
    const int n_r = ix.n_r[b];
    const int k = tk.v[b];
    const float neg_inf = -__builtin_huge_valf();
    if (n_r == 0) {
        if (threadIdx.x == 0) w.tau_lo[row] = neg_inf;
        return;
    }
    const int stride = sample_stride(n_r);
    const int ns = (n_r + stride - 1) / stride;
    // order statistic: about 2k * ns / |R| sampled tokens above, plus a margin
    const int c = (k == 0) ? 1 : static_cast<int>(ceilf(2.0f * k * ns / n_r)) + 8;
    if (c > ns) {   // the budget is a large share of R: every token is a candidate
        if (threadIdx.x == 0) w.tau_lo[row] = neg_inf;
        return;
    }
    stage_head_lut<kSelThreads>(lut_s, w.lut + static_cast<int64_t>(bg) * kLutRow * D.G, D.G, hh);
    __syncthreads();
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const uint4* codes = reinterpret_cast<const uint4*>(ix.codes) + base;
    const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * D.G;
    for (int s = threadIdx.x; s < ns; s += kSelThreads) {
        const int pos = s * stride;
        const int j = ix.pos_list[base + pos];
        float fs[1];
        fine_sum<1>(lut_s, codes[pos], fs);
        const float score = pq_logit(ix.norms[base + pos], coarse[j * D.G + hh], fs[0]);
        keys[s] = float_key(score);
    }
    __syncthreads();
    const SelectResult r = block_select_desc<kSelThreads>(
        [&](int i) { return keys[i]; }, [](int) { return true; }, ns, c, sh);
    if (threadIdx.x == 0) w.tau_lo[row] = key_float(r.key) + bias;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(Dims D, BatchInts tk, Index ix,
                                                             Work w, int force_fallback) {
    __shared__ float mass[kMaxLists];
    __shared__ float lut_s[kLutRow];
    __shared__ SelectScratch sh;
    const int tid = threadIdx.x;
    const int row = blockIdx.x;
    const int b = row / D.Hq;
    const int h = row % D.Hq;
    const int g = h / D.G;
    const int hh = h % D.G;
    const int bg = b * D.Hkv + g;
    const int n_r = ix.n_r[b];
    const int k = tk.v[b];
    const int nsub = (n_r + kSub - 1) / kSub;
    const int64_t rbase = static_cast<int64_t>(row) * D.rcap;
    const int64_t base = static_cast<int64_t>(bg) * D.rcap;
    const float neg_inf = -__builtin_huge_valf();

    // 1) candidate count; each thread owns a contiguous range of sub-chunks
    const int per = (nsub + kSelThreads - 1) / kSelThreads;
    const int sc0 = min(tid * per, nsub);
    const int sc1 = min(sc0 + per, nsub);
    const int32_t* cnt = w.cand_cnt + static_cast<int64_t>(row) * D.nsub_cap;
    int mine = 0;
    for (int sc = sc0; sc < sc1; ++sc) mine += cnt[sc];
    int total = 0;
    const int off = block_excl_scan<kSelThreads>(mine, total, sh);
    const bool fallback = force_fallback || (n_r > 0 && total < (k > 0 ? k : 1));

    if (!fallback) {
        // 2a) compact the row's candidates, position order
        int o = off;
        for (int sc = sc0; sc < sc1; ++sc) {
            const int c = cnt[sc];
            const int64_t src = rbase + static_cast<int64_t>(sc) * kSub;
            for (int i = 0; i < c; ++i, ++o) {
                w.comp_key[rbase + o] = float_key(w.cand_score[src + i]);
                w.comp_pos[rbase + o] = w.cand_pos[src + i];
            }
        }
    } else {
        // 2b) re-scan: every indexed token of the row is a candidate
        stage_head_lut<kSelThreads>(lut_s, w.lut + static_cast<int64_t>(bg) * kLutRow * D.G, D.G,
                                    hh);
        __syncthreads();
        const uint4* codes = reinterpret_cast<const uint4*>(ix.codes) + base;
        const float* coarse = w.coarse + static_cast<int64_t>(bg) * D.n_list * D.G;
        for (int pos = tid; pos < n_r; pos += kSelThreads) {
            const int j = ix.pos_list[base + pos];
            float fs[1];
            fine_sum<1>(lut_s, codes[pos], fs);
            const float s = pq_logit(ix.norms[base + pos], coarse[j * D.G + hh], fs[0]);
            w.comp_key[rbase + pos] = float_key(s);
            w.comp_pos[rbase + pos] = pos;
        }
        total = n_r;
    }
    __syncthreads();

    const uint32_t* ckey = w.comp_key + rbase;
    const int32_t* cpos = w.comp_pos + rbase;
    const int32_t* perm = ix.perm + base;

    // 3) the k-th largest key, and the token-id cut among equal keys
    uint32_t kth = 0xffffffffu;
    int tok_cut = 0x7fffffff;
    float shift = neg_inf;
    if (total > 0) {
        const SelectResult r = block_select_desc<kSelThreads>(
            [&](int i) { return ckey[i]; }, [](int) { return true; }, total, k > 0 ? k : 1, sh);
        shift = key_float(r.key);
        if (k > 0) {
            kth = r.key;
            const int need = k - r.count_above;
            if (r.count_equal > need) {
                const SelectResult t = block_select_desc<kSelThreads>(
                    [&](int i) { return ~static_cast<uint32_t>(perm[cpos[i]]); },
                    [&](int i) { return ckey[i] == kth; }, total, need, sh);
                tok_cut = static_cast<int>(~t.key);
            }
        }
    }

    // 4) emit T (candidate order) and the unselected-candidate masses per list
    for (int j = tid; j < D.n_list; j += kSelThreads) mass[j] = 0.0f;
    __syncthreads();
    int written = 0;
    int32_t* sel_tok = w.sel_tok + static_cast<int64_t>(row) * D.max_topk;
    int32_t* sel_pos = w.sel_pos + static_cast<int64_t>(row) * D.max_topk;
    for (int t0 = 0; t0 < total; t0 += kSelThreads) {
        const int i = t0 + tid;
        bool sel = false;
        int pos = 0, tok = -1;
        if (i < total) {
            const uint32_t key = ckey[i];
            pos = cpos[i];
            if (k > 0) {
                if (key > kth) {
                    sel = true;
                } else if (key == kth) {
                    tok = perm[pos];
                    sel = tok <= tok_cut;
                }
            }
            if (!sel) atomicAdd(&mass[ix.pos_list[base + pos]], __expf(key_float(key) - shift));
        }
        int tot = 0;
        const int o = block_excl_scan<kSelThreads>(sel ? 1 : 0, tot, sh);
        if (sel && written + o < k) {
            if (tok < 0) tok = perm[pos];
            sel_tok[written + o] = tok;
            sel_pos[written + o] = pos;
        }
        written += tot;
    }
    __syncthreads();
    float* cm = w.cand_mass + static_cast<int64_t>(row) * D.n_list;
    for (int j = tid; j < D.n_list; j += kSelThreads) cm[j] = mass[j];
    if (tid == 0) {
        w.row_shift[row] = shift;
        w.row_flag[row] = fallback ? 1 : 0;
    }
}

hipError_t launch_sample(const Dims& D, const BatchInts& tk, const Index& ix, const Work& w,
                         float bias, hipStream_t s) {
    hipLaunchKernelGGL(sample_kernel, dim3(D.B * D.Hq), dim3(kSelThreads), 0, s, D, tk, ix, w,
                       bias);
    return hipGetLastError();
}

hipError_t launch_select(const Dims& D, const BatchInts& tk, const Index& ix, const Work& w,
                         int force_fallback, hipStream_t s) {
    hipLaunchKernelGGL(select_kernel, dim3(D.B * D.Hq), dim3(kSelThreads), 0, s, D, tk, ix, w,
                       force_fallback);
    return hipGetLastError();
}

}  // namespace pqhsa
