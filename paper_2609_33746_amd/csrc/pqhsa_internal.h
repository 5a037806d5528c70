// Internal types and kernel launchers of libpqhsa (not part of the C ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pqhsa {

// --- tiling constants ------------------------------------------------------
constexpr int kHeadDim = 128;      // d

// The two product-quantizer layouts of the index (Section 3.1, Eq. 2).
// Pq8: 16 subspaces of 8 dimensions, 256 codewords, one byte per code
// (16 bytes per position). Pq4, the paper's own setting: 8 subspaces of 16
// dimensions, 16 codewords, two codes per byte (4 bytes per position; code m
// in bits 4m .. 4m + 3 of the word).
struct Pq8 {
    static constexpr int M = 16, K = 256, DSUB = 8, CODE_BYTES = 16, BITS = 8;
    static constexpr int LUT_ROW = M * K;   // fine-table entries per query head
    using Code = uint4;
};
struct Pq4 {
    static constexpr int M = 8, K = 16, DSUB = 16, CODE_BYTES = 4, BITS = 4;
    static constexpr int LUT_ROW = M * K;
    using Code = uint32_t;
};
constexpr int kLutRowMax = Pq8::LUT_ROW;
constexpr int kMaxBatch = 256;
constexpr int kMaxLists = 4096;

constexpr int kSub = 128;          // list-major positions per wave sub-chunk
constexpr int kScanWaves = 16;     // waves (sub-chunks) per scan workgroup
constexpr int kMaxSamples = 2048;  // sampled positions per row for the threshold
constexpr int kSelThreads = 1024;
constexpr int kSelCap = 12288;     // candidates of one row held in LDS by the select kernel
constexpr int kSelMaxSub = 1024;   // sub-chunks per row on the select kernel's fast path
constexpr int kSampleRun = 2;      // contiguous positions per sampled run
constexpr int kPosBits = 20;       // position / candidate word: list id << kPosBits | token id
constexpr uint32_t kPosMask = (1u << kPosBits) - 1u;
constexpr int kMaxSeq = 1 << kPosBits;
constexpr int kAttnRows = 128;     // exact-set rows per split, the larger of the two sizes
constexpr int kAttnRowsSmall = 64; // the split of small exact sets (see attn_rows_for)
constexpr int kBgLists = 64;       // lists per background workgroup
constexpr int kDenseRows = 2048;   // cache rows per dense split
constexpr int kPartStride = 132;   // floats per partial: m, Z, pad, pad, N[128]
constexpr int kMaxRowParts = 512;  // partials per row (exact splits + background chunks)
constexpr int kTailGrowth = 1024;  // tokens past the local window held exact between updates

// Optional events a launch records around its kernel's own execution
// (hipExtLaunchKernel), for per-kernel timing; null events record nothing.
struct KTiming {
    hipEvent_t start = nullptr, stop = nullptr;
};

// --- kernel arguments ----------------------------------------------------
struct Dims {
    int B, Hq, Hkv, G, n_list, n_sink, n_local;
    int rcap;       // per-(b, kv head) capacity of list-major arrays (= max_seq)
    int nsub_cap;   // ceil(rcap / kSub)
    int nseg_cap;   // n_list + nsub_cap
    int max_topk;
    int pq_bits;    // 8 (Pq8) or 4 (Pq4)
    int attn_rows;  // exact-set rows per split of the attend: kAttnRowsSmall or kAttnRows
    float inv_sqrt_d;
};

// Exact-set rows per attend split for a context: 64 when S, the local window
// and the largest budget hold at most 2048 rows (twice the splits spread a
// row's gathers over more CUs), else 128 (measured: one 128K sequence 56.4 ->
// 55.2 us, 16 sequences 245.7 -> 243.6 us; at a budget of 2621 the 64-row
// splits were slower, 40.5 -> 43.8 us in the attend).
__host__ __device__ inline int attn_rows_for(int n_sink, int n_local, int max_topk) {
    return n_sink + n_local + max_topk <= 2048 ? kAttnRowsSmall : kAttnRows;
}

// Compute units of the current device (0 if the runtime cannot say), read
// once per process; launch shapes that depend on how many workgroups run at
// once use it.
inline int device_cu_count() {
    static const int n_cu = [] {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        return n;
    }();
    return n_cu;
}

// One int per batch element, passed by value (top-k budgets, lengths).
struct BatchInts {
    int32_t v[kMaxBatch];
};

// The per-sequence integers every decode kernel needs, passed by value so
// that no kernel starts with a dependent load: k_b, |R_b| and |L_b|, the
// exact tail after R_b (N_b = n_sink + |R_b| + |L_b|; |L_b| = n_local right
// after an index prepare or update, up to n_local + kTailGrowth between them).
struct BatchArgs {
    int32_t topk[kMaxBatch];
    int32_t n_r[kMaxBatch];
    int32_t n_tail[kMaxBatch];
};

// Prepared index (list-major), owned by the context.
struct Index {
    const uint8_t* codes;      // [B, Hkv, rcap, M]
    const float* norms;        // [B, Hkv, rcap]
    const int32_t* perm;       // [B, Hkv, rcap] token id of each position
    const uint32_t* pos_word;  // [B, Hkv, rcap] list id << kPosBits | token id of each position
    const int32_t* loff;       // [B, Hkv, n_list + 1] list starts
    const float* centroids;    // [B, Hkv, n_list, d]
    const float* codebooks;    // [B, Hkv, M, K, d/M]
    const float* means;        // [B, Hkv, n_list, d]
    const float* glob_mean;    // [B, Hkv, d] sum_j |R_j| v_bar_j / |R_b| (variant C)
    const int32_t* n_seq;      // [B]
    const int32_t* n_r;        // [B] |R_b|
    // the threshold sample's positions, gathered once per prepare or update
    // (sample_position) so that the prologue reads them contiguously
    const uint8_t* samp_codes;  // [B, Hkv, kMaxSamples] codes (16 bytes a slot)
    const float* samp_norms;    // [B, Hkv, kMaxSamples]
    const int32_t* samp_list;   // [B, Hkv, kMaxSamples] list id
};

// The s-th position of the threshold sample of a row with n_r > 0 indexed
// tokens: runs of kSampleRun positions, rs = n_r / nrun apart, clipped at
// the next run. Returns false when s lies past the sample (sample count:
// nrun * run_len).
struct SampleRuns {
    int nrun, rs, run_len;
};
__host__ __device__ inline SampleRuns sample_runs(int n_r) {
    const int nrun = min(kMaxSamples / kSampleRun, (n_r + kSampleRun - 1) / kSampleRun);
    const int rs = n_r / nrun;
    return SampleRuns{nrun, rs, min(kSampleRun, rs)};
}
__host__ __device__ inline bool sample_position(const SampleRuns& sr, int s, int n_r, int& pos) {
    const int run = s / kSampleRun;
    const int within = s % kSampleRun;
    pos = run * sr.rs + within;
    return run < sr.nrun && within < sr.run_len && pos < n_r;
}

// Decode workspace, owned by the context.
struct Work {
    float* lut;          // [B, Hkv, M, K, G]   (q^(m) . p_{m,z}) / sqrt(d)
    float* lut_head;     // [B, Hq, M, K]       the same entries, head-major
    uint32_t* lut_flag;  // [B, Hkv, prologue_parts] epoch of the last call each LUT part finished
    uint32_t* epoch;     // [B, Hkv] decode calls completed on this workspace (advanced by the merge)
    float* coarse;       // [B, Hkv, n_list, G] (q . c_j) / sqrt(d)
    float* tau_lo;       // [B, Hq] candidate threshold
    float* tau_hi;       // [B, Hq] largest sampled score (-inf when not sampled)
    uint2* cand;         // [B, Hq, rcap] candidates compacted per sub-chunk: (score bits,
                         //   list id << kPosBits | list-major position)
    int32_t* cand_cnt;   // [B, Hq, nsub_cap]
    float* seg_sum;      // [B, Hkv, nseg_cap, G] below-threshold masses; the pair
                         //   (list j, sub-chunk s) uses segment j + s
    uint32_t* comp_key;  // [B, Hq, rcap] contiguous candidates (order keys)
    int32_t* comp_pos;   // [B, Hq, rcap] (same packing as the candidate word)
    int32_t* sel_tok;    // [B, Hq, max_topk] token ids of T
    float* cand_mass;    // [B, Hq, n_list] sum over the list's unselected candidates of
                         //   exp(l~ - shift)
    float* row_shift;    // [B, Hq] shift of the background masses
    int32_t* row_flag;   // [B, Hq] 1 when the row took the re-scan path
    float* partial;      // [B, Hq, nsplit_max + n_bgc, kPartStride]
    float* bx_w;         // [B, Hq, n_list] variant Bx: M_j / |B n R_j| (0 when no member
                         //   of list j is unselected)
    float* bx_wsel;      // [B, Hq, max_topk] variant Bx: bx_w of the list of each entry of T
    // A call whose budgets and lengths are device data: the caller's N_b and
    // k_b (dev_lens, dev_topk), and the call's clamped per-sequence integers
    // (ba_dev), written by the prologue for the later kernels. All null when
    // the integers travel by value in BatchArgs.
    BatchArgs* ba_dev;
    const int32_t* dev_lens;
    const int32_t* dev_topk;
};

// The integers of batch element b in a device-argument call, from |R_b| of
// the prepared index and the caller's N_b and k_b: k_b clamped into
// [0, min(|R_b|, max_topk)], the tail N_b - n_sink - |R_b| into
// [0, n_local + kTailGrowth] and into the cache. Device data are not
// validated, so clamping is what keeps every kernel inside its buffers.
struct SeqArgs {
    int topk, n_r, n_tail;
};
__device__ __forceinline__ SeqArgs clamp_seq_args(const Dims& D, int n_r, int seq_len, int topk) {
    const int tail_cap = min(D.n_local + kTailGrowth, D.rcap - D.n_sink - n_r);
    return SeqArgs{min(max(topk, 0), min(n_r, D.max_topk)), n_r,
                   min(max(seq_len - D.n_sink - n_r, 0), tail_cap)};
}

// k_b, |R_b| and the tail |L_b| of a call: from the kernel argument, or
// (kDev, a separate instantiation of each kernel) from device memory when the
// call's budgets and lengths are device data. A runtime choice between the
// two made the compiler merge them into one generic load that waits for
// memory at kernel start (1.3 us per call at 128K).
template <bool kDev>
__device__ __forceinline__ int arg_topk(const BatchArgs& ba, const Work& w, int b) {
    if constexpr (kDev) return w.ba_dev->topk[b];
    else return ba.topk[b];
}
template <bool kDev>
__device__ __forceinline__ int arg_n_r(const BatchArgs& ba, const Work& w, int b) {
    if constexpr (kDev) return w.ba_dev->n_r[b];
    else return ba.n_r[b];
}
template <bool kDev>
__device__ __forceinline__ int arg_n_tail(const BatchArgs& ba, const Work& w, int b) {
    if constexpr (kDev) return w.ba_dev->n_tail[b];
    else return ba.n_tail[b];
}

// The caller's KV cache. Contiguous: token t of (b, g) at b sb + g sh + t sn
// elements. Paged (bt != null): at bt[b max_blocks + t >> page_shift] sb +
// g sh + (t & (2^page_shift - 1)) sn, sb then being the page stride.
struct KV {
    const void* q;
    const void* k;
    const void* v;
    int64_t sb, sh, sn;   // element strides of (b or page, kv head, token)
    int bf16;
    const int32_t* bt = nullptr;   // [B, max_blocks] page of each logical block
    int max_blocks = 0;
    int page_shift = 0;
};

// Element offset of token t of (b, g) in the cache (t >= 0).
__device__ __forceinline__ int64_t kv_row(const KV& kv, int b, int g, int t) {
    if (kv.bt) {
        const int pg = kv.bt[static_cast<int64_t>(b) * kv.max_blocks + (t >> kv.page_shift)];
        return pg * kv.sb + g * kv.sh + (t & ((1 << kv.page_shift) - 1)) * kv.sn;
    }
    return b * kv.sb + g * kv.sh + t * kv.sn;
}

// --- launchers (each returns the launch status) -----------------------
// Kernel attributes (large dynamic LDS) for the current device; called once
// per context creation.
hipError_t configure_select();

// LUT workgroups per (b, kv head) in the prologue: fine parts (8 for Pq8,
// 2 subspaces each; 1 for Pq4) plus one coarse part per kCoarseLists lists.
__host__ __device__ inline int prologue_fine_parts(int pq_bits) { return pq_bits == 4 ? 1 : 8; }
constexpr int kCoarseLists = 64;   // lists per coarse LUT workgroup of the prologue
__host__ __device__ inline int prologue_parts(int n_list, int pq_bits) {
    return prologue_fine_parts(pq_bits) + (n_list + kCoarseLists - 1) / kCoarseLists;
}
hipError_t launch_prologue(const Dims& D, const BatchArgs& ba, const KV& kv, const Index& ix,
                           const Work& w, float bias, hipStream_t s,
                           const KTiming& tm = KTiming{});
// nwg = scan workgroups per (batch element, KV head): enough for the longest R_b
hipError_t launch_scan(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w, int nwg,
                       hipStream_t s, const KTiming& tm = KTiming{});
// bx: variant Bx, whose per-list weights bx_w and per-entry weights bx_wsel
// the select forms beside T
hipError_t launch_select(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                         int force_fallback, bool bx, hipStream_t s, const KTiming& tm = KTiming{});
// variant: the background term, a PQHSA_VARIANT_* value. nsplit: exact-set
// splits launched per row (enough for this call's rows); nsplit_max: the
// splits per row the partial buffer holds (its layout).
hipError_t launch_attend(const Dims& D, const BatchArgs& ba, const KV& kv, const Index& ix,
                         const Work& w, int nsplit, int nsplit_max, int variant, hipStream_t s,
                         const KTiming& tm = KTiming{});
hipError_t launch_merge(const Dims& D, const BatchArgs& ba, const Work& w, float* out,
                        int nsplit_max, int variant, hipStream_t s, const KTiming& tm = KTiming{});
hipError_t launch_dense(const Dims& D, const KV& kv, const BatchInts& lens, float* partial,
                        float* out, int nsplit_max, hipStream_t s);
// The fixed scratch array of the entry point that allocates nothing: its size,
// and its device address on the current device (looked up on the first call
// per device, then kept).
size_t static_scratch_bytes();
hipError_t static_scratch(void** ptr);
// the token-weighted mean of the list means per (b, g): the global value
// mean over R_b of variant C
hipError_t launch_glob_mean(const Dims& D, const Index& ix, float* glob, hipStream_t s);
// The coarse assignment of the build on the matrix cores: the nearest center
// of every token of R_b (ids_tm) and its squared distance (dist_c, or null).
hipError_t launch_assign(const Dims& D, const BatchInts& lo, const BatchInts& hi, int max_n,
                         const KV& kv, const float* centroids, int32_t* ids_tm, float* dist_c,
                         hipStream_t s);
// The codeword search of the build on the matrix cores, for tokens whose
// lists are in ids_tm: norms, codes and the chosen distances (dist_f or null).
hipError_t launch_subspace(const Dims& D, const BatchInts& lo, const BatchInts& hi, int max_n,
                           const KV& kv, const float* centroids, const float* codebooks,
                           const int32_t* ids_tm, uint8_t* codes_tm, float* norms_tm, float* dist_f,
                           hipStream_t s);
// the update's encoding of the tokens leaving the window: one workgroup per token
hipError_t launch_encode_update(const Dims& D, const BatchInts& lo, const BatchInts& hi,
                                int max_new, const KV& kv, const float* centroids,
                                const float* codebooks, int32_t* ids_tm, uint8_t* codes_tm,
                                float* norms_tm, hipStream_t s);
// index build steps (k-means over the tokens [lo[b], hi[b]) of each (b, kv head))
struct BuildBufs {
    int32_t* order;      // [problems, rcap] tokens grouped by center, in id order within a center
    int32_t* offs;       // [problems, n_centers + 1]
    float* dist_c;       // [B, Hkv, rcap]
    float* dist_f;       // [B, Hkv, rcap, M]
    int32_t* seg_hist;   // [problems, segments of 4096 tokens, keys] counts, then first positions
                         //   (problems with at most 1024 keys)
};
constexpr int kBuildSegTok = 4096;   // tokens per segment of the build's grouping
// kind: 0 coarse centers over directions, 1 codewords over residual slices,
// 2 list means over values
// The stable grouping of launch_group for problems of at most 1024 keys,
// over segments of kBuildSegTok tokens: order [problems, rcap] (tokens by key,
// in id order within a key) and offs [problems, keys + 1]; seg_hist holds
// problems x ceil(max |R_b| / kBuildSegTok) x keys ints of scratch.
hipError_t launch_group_segments(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                                 const int32_t* ids_tm, const uint8_t* codes_tm, int32_t* seg_hist,
                                 int32_t* order, int32_t* offs, hipStream_t s);
hipError_t launch_group(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                        const int32_t* ids_tm, const uint8_t* codes_tm, const BuildBufs& bb,
                        hipStream_t s);
hipError_t launch_centers(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                          const KV& kv, const int32_t* ids_tm, const float* norms_tm,
                          const float* centroids, const BuildBufs& bb, float* out, hipStream_t s);
hipError_t launch_init_centers(const Dims& D, int kind, const KV& kv, const int32_t* init,
                               const int32_t* ids_tm, const float* norms_tm, const float* centroids,
                               float* out, hipStream_t s);
hipError_t launch_reseed(const Dims& D, const BatchInts& lo, const BatchInts& hi, int kind,
                         const KV& kv, const int32_t* ids_tm, const float* norms_tm,
                         const float* centroids, const BuildBufs& bb, float* out, hipStream_t s);

// the list-major rebuild after an update's encode pass (lo, hi as there):
// new list offsets, per-list shifts [B, Hkv, n_list] and the new perm /
// pos_word in the *_new buffers (which must not alias the old ones); n_r,
// n_seq, the float64 list value sums and the list means (from the values
// in kv) updated in place
// The list-major layout of R_b = tokens [lo_b, hi_b) built from the
// token-major list ids on the device: a stable counting sort per (b, kv
// head), lists in increasing id, tokens in increasing id within a list.
// zero_loff: [B, Hkv, n_list + 1] zeros. bad: one word set to all ones
// beforehand; receives the smallest flat index of an id outside [0, n_list).
// scratch (scratch_ints ints, may be null): with up to 1024 lists and room for
// the per-segment counts, the sort runs as the build's segmented grouping
// over many workgroups per (b, g); otherwise one workgroup per (b, g).
hipError_t launch_sort_lists(const Dims& D, const BatchInts& lo, const BatchInts& hi, int max_n,
                             const int32_t* ids_tm, const int32_t* zero_loff, int32_t* loff,
                             int32_t* shift, int32_t* perm, uint32_t* pos_word, int32_t* n_r_dev, int32_t* n_seq_dev, unsigned long long* bad,
                             int32_t* scratch, size_t scratch_ints, hipStream_t s);
hipError_t launch_update_lists(const Dims& D, const BatchInts& lo, const BatchInts& hi,
                               const KV& kv, const int32_t* ids_tm, const int32_t* old_loff,
                               const int32_t* perm_old, const uint32_t* pos_old, int32_t* new_loff,
                               int32_t* shift, int32_t* perm_new, uint32_t* pos_new,
                               int32_t* n_r_dev, int32_t* n_seq_dev,
                               float* means, double* sums, hipStream_t s);
// float64 value sums of the lists, |R_j| v_bar_j, for later updates
hipError_t launch_init_sums(const Dims& D, const int32_t* loff, const float* means, double* sums,
                            hipStream_t s);
// The threshold sample's codes, norms and list ids per (b, kv head), from the
// list-major index (after every prepare and update).
hipError_t launch_sample_slab(const Dims& D, const Index& ix, uint8_t* samp_codes, float* samp_norms,
                              int32_t* samp_list, hipStream_t s);
hipError_t launch_prepare_gather(const Dims& D, const uint8_t* codes_in, const float* norms_in,
                                 const Index& ix, uint8_t* codes_out, float* norms_out,
                                 hipStream_t s);
hipError_t launch_debug(const Dims& D, const BatchArgs& ba, const Index& ix, const Work& w,
                        int32_t* selected, int32_t* unselected, float* scores,
                        hipStream_t s);

}  // namespace pqhsa
