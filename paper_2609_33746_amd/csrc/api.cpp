// Host side of libpqhsa: argument validation, context and workspace
// management, index preparation and the stream-ordered launch sequence of a
// decode step. Every numeric step of the operator runs in the HIP kernels of
// this library; the host only validates, reorders index metadata at prepare
// time and enqueues work.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pqhsa.h"
#include "pqhsa_internal.h"

using namespace pqhsa;

namespace {

thread_local std::string g_create_error;

constexpr int kStages = 5;

}  // namespace

struct pqhsa_ctx {
    pqhsa_shape shape{};
    Dims D{};
    int device = 0;
    std::string err;
    std::vector<void*> allocs;

    // prepared index (device)
    bool prepared = false;
    std::vector<int32_t> seq_lens, n_r;   // N_b and |R_b| of the index
    std::vector<int32_t> cur_len;         // current cache lengths (>= seq_lens; the tail is exact)
    uint8_t* codes = nullptr;
    float* norms = nullptr;
    uint8_t* samp_codes = nullptr;   // the threshold sample (Index::samp_*)
    float* samp_norms = nullptr;
    int32_t* samp_list = nullptr;
    int32_t* perm = nullptr;
    uint32_t* pos_word = nullptr;
    int32_t* loff = nullptr;
    float* centroids = nullptr;
    float* codebooks = nullptr;
    float* means = nullptr;
    float* glob_mean = nullptr;   // [B, Hkv, d] for variant C
    double* mean_sums = nullptr;  // [B, Hkv, n_list, d] float64 value sums of the lists (updates)
    // token-major copy of the index, the source of every list-major rebuild
    int32_t* ids_tm = nullptr;       // [B, Hkv, rcap] list id of each token
    uint8_t* codes_tm = nullptr;     // [B, Hkv, rcap, M] one code per byte
    float* norms_tm = nullptr;       // [B, Hkv, rcap]
    // the other half of the double-buffered list-major arrays (an update
    // builds the new layout there, then the two halves swap)
    int32_t* perm_alt = nullptr;
    uint32_t* pos_alt = nullptr;
    int32_t* loff_alt = nullptr;
    int32_t* shift = nullptr;        // [B, Hkv, n_list] per-list position shift of an update
    int32_t* n_seq_dev = nullptr;
    int32_t* n_r_dev = nullptr;
    unsigned long long* bad_id = nullptr;   // first invalid list id found by a prepare
    BatchArgs* ba_dev = nullptr;   // a device-argument decode's per-sequence integers
    int scan_nwg = 0;   // scan workgroups per (b, kv head)

    // workspace
    Work w{};
    int nsplit_max = 0;
    float* dense_partial = nullptr;
    int dense_nsplit = 0;
    size_t codebook_floats = 0;   // per (b, kv head): K * d

    // options
    int force_fallback = 0;
    int timing = 0;
    float bias = 0.0f;
    int variant = PQHSA_VARIANT_B;
    hipEvent_t ev[2 * kStages]{};   // start and stop of each stage's kernel
    bool events_made = false;
    bool timed_valid = false;

    Index index() const {
        Index ix;
        ix.codes = codes;
        ix.norms = norms;
        ix.perm = perm;
        ix.pos_word = pos_word;
        ix.loff = loff;
        ix.centroids = centroids;
        ix.codebooks = codebooks;
        ix.means = means;
        ix.glob_mean = glob_mean;
        ix.n_seq = n_seq_dev;
        ix.n_r = n_r_dev;
        ix.samp_codes = samp_codes;
        ix.samp_norms = samp_norms;
        ix.samp_list = samp_list;
        return ix;
    }
};

namespace {

pqhsa_status fail(pqhsa_ctx* c, pqhsa_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    if (c) c->err = buf;
    else g_create_error = buf;
    return st;
}

pqhsa_status hip_fail(pqhsa_ctx* c, hipError_t e, const char* what) {
    return fail(c, PQHSA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

template <typename T>
hipError_t dev_alloc(pqhsa_ctx* c, T** p, size_t count) {
    void* raw = nullptr;
    const size_t bytes = std::max<size_t>(count * sizeof(T), 256);
    hipError_t e = hipMalloc(&raw, bytes);
    if (e != hipSuccess) return e;
    c->allocs.push_back(raw);
    *p = static_cast<T*>(raw);
    return hipSuccess;
}

pqhsa_status check_shape(const pqhsa_shape* s) {
    if (!s) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "shape is NULL");
    if (s->batch < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->max_seq < 1)
        return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT,
                    "batch, n_q_heads, n_kv_heads and max_seq must be positive");
    if (s->n_q_heads % s->n_kv_heads)
        return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "n_q_heads must be a multiple of n_kv_heads");
    if (s->n_sink < 0 || s->n_local < 0 || s->n_sink + s->n_local > s->max_seq)
        return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "need 0 <= n_sink, n_local and n_sink + n_local <= max_seq");
    if (s->max_topk < 0 || s->max_topk > s->max_seq)
        return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "need 0 <= max_topk <= max_seq");
    if (s->n_list < 1) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "n_list must be positive");
    if (s->kv_dtype != PQHSA_F32 && s->kv_dtype != PQHSA_BF16)
        return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "kv_dtype must be PQHSA_F32 or PQHSA_BF16");
    if (s->head_dim != kHeadDim) return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "head_dim must be 128");
    if (!((s->pq_m == Pq8::M && s->pq_ksub == Pq8::K) || (s->pq_m == Pq4::M && s->pq_ksub == Pq4::K)))
        return fail(nullptr, PQHSA_ERR_UNSUPPORTED,
                    "(pq_m, pq_ksub) must be (16, 256) or (8, 16)");
    const int G = s->n_q_heads / s->n_kv_heads;
    if (G != 1 && G != 2 && G != 4 && G != 8)
        return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "GQA group size must be 1, 2, 4 or 8");
    if (s->batch > kMaxBatch) return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "batch must be <= 256");
    if (s->n_list > kMaxLists) return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "n_list must be <= 4096");
    if (s->max_seq > kMaxSeq) return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "max_seq must be <= 2^20");
    {
        // partials per row: splits of the exact set plus background chunks
        const int rows = attn_rows_for(s->n_sink, s->n_local, s->max_topk);
        const int nsplit = std::max((s->n_sink + s->n_local + kTailGrowth + s->max_topk + rows - 1) / rows, 1);
        const int nbgc = (s->n_list + kBgLists - 1) / kBgLists;
        if (nsplit + nbgc > kMaxRowParts)
            return fail(nullptr, PQHSA_ERR_UNSUPPORTED,
                        "n_sink + n_local + max_topk must be <= %d for n_list = %d",
                        (kMaxRowParts - nbgc) * kAttnRows - kTailGrowth, s->n_list);
    }
    return PQHSA_OK;
}

pqhsa_status check_device(pqhsa_ctx* c) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(c, e, "hipGetDevice");
    if (dev != c->device)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "current device %d is not the context's device %d", dev,
                    c->device);
    return PQHSA_OK;
}

// The cache pointers and strides of a call; errors go to c (or, with c null,
// to the thread's context-free message).
pqhsa_status check_kv_dtype(pqhsa_ctx* c, int kv_dtype, const void* q, const void* k,
                            const void* v, const int64_t* strides, const void* out, KV* kv) {
    if (!q || !k || !v || !out || !strides)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "q, k_cache, v_cache, kv_strides and out must be non-NULL");
    const int64_t sb = strides[0], sh = strides[1], sn = strides[2];
    if (sb < 0 || sh < 0 || sn < kHeadDim)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT,
                    "kv_strides must be non-negative with a token stride >= head_dim");
    const int esz = kv_dtype == PQHSA_BF16 ? 2 : 4;
    if ((sb * esz) % 16 || (sh * esz) % 16 || (sn * esz) % 16 ||
        reinterpret_cast<uintptr_t>(k) % 16 || reinterpret_cast<uintptr_t>(v) % 16 ||
        reinterpret_cast<uintptr_t>(q) % 16)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "q, k_cache, v_cache and their strides must be 16-byte aligned");
    kv->q = q;
    kv->k = k;
    kv->v = v;
    kv->sb = sb;
    kv->sh = sh;
    kv->sn = sn;
    kv->bf16 = kv_dtype == PQHSA_BF16;
    return PQHSA_OK;
}

pqhsa_status check_kv(pqhsa_ctx* c, const void* q, const void* k, const void* v,
                      const int64_t* strides, const void* out, KV* kv) {
    return check_kv_dtype(c, c->shape.kv_dtype, q, k, v, strides, out, kv);
}

// A paged cache: the strides are those of (page, kv head, token in page);
// page_size a power of two, and the block table long enough for the longest
// prepared sequence.
pqhsa_status check_pages(pqhsa_ctx* c, const int32_t* block_table, int32_t max_blocks,
                         int32_t page_size, KV* kv) {
    if (!block_table) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "block_table is NULL");
    if (page_size < 1 || page_size > (1 << 20) || (page_size & (page_size - 1)))
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "page_size %d is not a power of two in [1, 2^20]",
                    page_size);
    int n_max = 0;
    for (int n : c->cur_len) n_max = std::max(n_max, n);
    if (max_blocks < 1 || static_cast<int64_t>(max_blocks) * page_size < n_max)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT,
                    "max_blocks %d x page_size %d does not cover the longest sequence (%d tokens)",
                    max_blocks, page_size, n_max);
    kv->bt = block_table;
    kv->max_blocks = max_blocks;
    kv->page_shift = __builtin_ctz(static_cast<unsigned>(page_size));
    return PQHSA_OK;
}

}  // namespace

extern "C" {

const char* pqhsa_status_string(pqhsa_status st) {
    switch (st) {
        case PQHSA_OK: return "ok";
        case PQHSA_ERR_INVALID_ARGUMENT: return "invalid argument";
        case PQHSA_ERR_UNSUPPORTED: return "unsupported";
        case PQHSA_ERR_HIP: return "HIP runtime error";
        case PQHSA_ERR_OUT_OF_MEMORY: return "out of memory";
        case PQHSA_ERR_NOT_PREPARED: return "index not prepared";
        default: return "unknown status";
    }
}

const char* pqhsa_last_error(const pqhsa_ctx* ctx) {
    return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

void pqhsa_destroy(pqhsa_ctx* ctx) {
    if (!ctx) return;
    if (ctx->events_made)
        for (auto& e : ctx->ev) (void)hipEventDestroy(e);
    for (void* p : ctx->allocs) (void)hipFree(p);
    delete ctx;
}

pqhsa_status pqhsa_create(const pqhsa_shape* shape, pqhsa_ctx** out) {
    g_create_error.clear();
    if (!out) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    pqhsa_status st = check_shape(shape);
    if (st != PQHSA_OK) return st;

    pqhsa_ctx* c = new (std::nothrow) pqhsa_ctx();
    if (!c) return fail(nullptr, PQHSA_ERR_OUT_OF_MEMORY, "host allocation failed");
    c->shape = *shape;
    hipError_t e = hipGetDevice(&c->device);
    if (e == hipSuccess) e = configure_select();
    if (e != hipSuccess) {
        delete c;
        return fail(nullptr, PQHSA_ERR_HIP, "device set-up: %s", hipGetErrorString(e));
    }
    Dims& D = c->D;
    D.B = shape->batch;
    D.Hq = shape->n_q_heads;
    D.Hkv = shape->n_kv_heads;
    D.G = D.Hq / D.Hkv;
    D.n_list = shape->n_list;
    D.n_sink = shape->n_sink;
    D.n_local = shape->n_local;
    D.rcap = shape->max_seq;
    D.nsub_cap = (D.rcap + kSub - 1) / kSub;
    D.nseg_cap = D.n_list + D.nsub_cap;
    D.max_topk = std::max(shape->max_topk, 1);
    D.attn_rows = attn_rows_for(D.n_sink, D.n_local, shape->max_topk);
    D.pq_bits = shape->pq_m == Pq4::M ? Pq4::BITS : Pq8::BITS;
    D.inv_sqrt_d = static_cast<float>(1.0 / std::sqrt(static_cast<double>(kHeadDim)));

    const size_t B = D.B, Hq = D.Hq, Hkv = D.Hkv, G = D.G, L = D.n_list, rc = D.rcap;
    const size_t BG = B * Hkv, BQ = B * Hq;
    c->nsplit_max = (D.n_sink + D.n_local + kTailGrowth + shape->max_topk + D.attn_rows - 1) / D.attn_rows;
    if (c->nsplit_max < 1) c->nsplit_max = 1;
    const int n_bgc = (D.n_list + kBgLists - 1) / kBgLists;
    c->dense_nsplit = (D.rcap + kDenseRows - 1) / kDenseRows;

    Work& w = c->w;
    hipError_t ea = hipSuccess;
    auto A = [&](hipError_t r) { if (ea == hipSuccess) ea = r; };
    const size_t code_bytes = D.pq_bits == 4 ? Pq4::CODE_BYTES : Pq8::CODE_BYTES;
    const size_t lut_row = D.pq_bits == 4 ? Pq4::LUT_ROW : Pq8::LUT_ROW;
    const size_t codebook_floats = (D.pq_bits == 4 ? Pq4::K : Pq8::K) * static_cast<size_t>(kHeadDim);
    c->codebook_floats = codebook_floats;
    A(dev_alloc(c, &c->codes, BG * rc * code_bytes));
    A(dev_alloc(c, &c->norms, BG * rc));
    A(dev_alloc(c, &c->perm, BG * rc));
    A(dev_alloc(c, &c->pos_word, BG * rc));
    A(dev_alloc(c, &c->loff, BG * (L + 1)));
    A(dev_alloc(c, &c->centroids, BG * L * kHeadDim));
    A(dev_alloc(c, &c->codebooks, BG * codebook_floats));
    A(dev_alloc(c, &c->means, BG * L * kHeadDim));
    A(dev_alloc(c, &c->glob_mean, BG * kHeadDim));
    A(dev_alloc(c, &c->mean_sums, BG * L * kHeadDim));
    A(dev_alloc(c, &c->ids_tm, BG * rc));
    A(dev_alloc(c, &c->codes_tm, BG * rc * static_cast<size_t>(shape->pq_m)));
    A(dev_alloc(c, &c->samp_codes, BG * kMaxSamples * 16));
    A(dev_alloc(c, &c->samp_norms, BG * kMaxSamples));
    A(dev_alloc(c, &c->samp_list, BG * kMaxSamples));
    A(dev_alloc(c, &c->norms_tm, BG * rc));
    A(dev_alloc(c, &c->perm_alt, BG * rc));
    A(dev_alloc(c, &c->pos_alt, BG * rc));
    A(dev_alloc(c, &c->loff_alt, BG * (L + 1)));
    A(dev_alloc(c, &c->shift, BG * L));
    A(dev_alloc(c, &c->n_seq_dev, B));
    A(dev_alloc(c, &c->n_r_dev, B));
    A(dev_alloc(c, &c->bad_id, 1));
    A(dev_alloc(c, &c->ba_dev, 1));
    A(dev_alloc(c, &w.lut, BG * lut_row * G));
    A(dev_alloc(c, &w.coarse, BG * L * G + 16));   // + 16: whole float4 reads at the end
    A(dev_alloc(c, &w.lut_head, BQ * lut_row));
    const size_t lut_parts = BG * prologue_parts(D.n_list, D.pq_bits);
    A(dev_alloc(c, &w.lut_flag, lut_parts));
    A(dev_alloc(c, &w.epoch, BG));
    if (ea == hipSuccess) ea = hipMemset(w.lut_flag, 0, lut_parts * sizeof(uint32_t));
    if (ea == hipSuccess) ea = hipMemset(w.epoch, 0, BG * sizeof(uint32_t));
    A(dev_alloc(c, &w.tau_lo, BQ));
    A(dev_alloc(c, &w.tau_hi, BQ));
    A(dev_alloc(c, &w.cand, BQ * rc));
    A(dev_alloc(c, &w.cand_cnt, BQ * D.nsub_cap));
    A(dev_alloc(c, &w.seg_sum, BG * D.nseg_cap * G));
    A(dev_alloc(c, &w.comp_key, BQ * rc));
    A(dev_alloc(c, &w.comp_pos, BQ * rc));
    A(dev_alloc(c, &w.sel_tok, BQ * D.max_topk));
    A(dev_alloc(c, &w.cand_mass, BQ * L));
    A(dev_alloc(c, &w.bx_w, BQ * L));
    A(dev_alloc(c, &w.bx_wsel, BQ * D.max_topk));
    A(dev_alloc(c, &w.row_shift, BQ));
    A(dev_alloc(c, &w.row_flag, BQ));
    A(dev_alloc(c, &w.partial, BQ * (c->nsplit_max + n_bgc) * kPartStride));
    A(dev_alloc(c, &c->dense_partial, BQ * c->dense_nsplit * kPartStride));
    if (ea != hipSuccess) {
        const bool oom = ea == hipErrorOutOfMemory || ea == hipErrorMemoryAllocation;
        char msg[256];
        snprintf(msg, sizeof(msg), "device allocation failed: %s", hipGetErrorString(ea));
        pqhsa_destroy(c);
        return fail(nullptr, oom ? PQHSA_ERR_OUT_OF_MEMORY : PQHSA_ERR_HIP, "%s", msg);
    }
    *out = c;
    return PQHSA_OK;
}

// Rebuild the list-major layout of every (b, kv head) from the token-major
// index (ids_tm, codes_tm, norms_tm) for sequence lengths `lens`, on the
// device: a check of the list ids, a stable counting sort of R_b by list id
// (lists in increasing id, tokens in increasing id within a list), the
// gather of codes and norms, the global value means and the list sums.
// Synchronises `stream`; fails (and leaves the context unprepared) when a
// list id of R lies outside [0, n_list).
static pqhsa_status relayout(pqhsa_ctx* c, const std::vector<int32_t>& lens, hipStream_t stream) {
    const Dims& D = c->D;
    const int B = D.B, Hkv = D.Hkv, L = D.n_list;
    const size_t rc = D.rcap;
    const size_t BG = static_cast<size_t>(B) * Hkv;
    std::vector<int32_t> nr(B);
    BatchInts lo{}, hi{};
    int max_n = 0;
    for (int b = 0; b < B; ++b) {
        nr[b] = lens[b] - D.n_sink - D.n_local;
        lo.v[b] = D.n_sink;
        hi.v[b] = D.n_sink + nr[b];
        max_n = std::max(max_n, nr[b]);
    }
    c->prepared = false;
    // the empty index the sort merges R into
    hipError_t e = hipMemsetAsync(c->loff_alt, 0, BG * (L + 1) * sizeof(int32_t), stream);
    if (e == hipSuccess) e = hipMemsetAsync(c->bad_id, 0xff, sizeof(unsigned long long), stream);
    if (e == hipSuccess)
        e = launch_sort_lists(D, lo, hi, max_n, c->ids_tm, c->loff_alt, c->loff, c->shift, c->perm,
                              c->pos_word, c->n_r_dev, c->n_seq_dev, c->bad_id,
                              reinterpret_cast<int32_t*>(c->w.comp_key),
                              static_cast<size_t>(D.B) * D.Hq * rc, stream);
    if (e != hipSuccess) return hip_fail(c, e, "launching the list-major sort");
    e = launch_prepare_gather(D, c->codes_tm, c->norms_tm, c->index(), c->codes, c->norms, stream);
    if (e == hipSuccess)
        e = launch_sample_slab(D, c->index(), c->samp_codes, c->samp_norms, c->samp_list, stream);
    if (e != hipSuccess) return hip_fail(c, e, "launching the index gather");
    e = launch_glob_mean(D, c->index(), c->glob_mean, stream);
    if (e == hipSuccess) e = launch_init_sums(D, c->loff, c->means, c->mean_sums, stream);
    if (e != hipSuccess) return hip_fail(c, e, "launching the global value mean and list sums");
    unsigned long long bad = 0;
    e = hipMemcpyAsync(&bad, c->bad_id, sizeof(bad), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(c, e, "preparing the index");
    if (bad != ~0ull) {
        int32_t value = 0;
        e = hipMemcpy(&value, c->ids_tm + bad, sizeof(value), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(c, e, "reading an invalid list id");
        const size_t bg = bad / rc;
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "list_ids[%d][%d][%d] = %d outside [0, n_list = %d)",
                    static_cast<int>(bg / Hkv), static_cast<int>(bg % Hkv), static_cast<int>(bad % rc),
                    value, L);
    }
    c->seq_lens = lens;
    c->cur_len = lens;
    c->n_r = nr;
    int nr_max = 0;
    for (int b = 0; b < B; ++b) nr_max = std::max(nr_max, nr[b]);
    c->scan_nwg = (nr_max + kScanWaves * kSub - 1) / (kScanWaves * kSub);
    c->prepared = true;
    return PQHSA_OK;
}


pqhsa_status pqhsa_index_prepare(pqhsa_ctx* c, const int32_t* seq_lens, const int32_t* list_ids,
                                 const uint8_t* codes, const float* norms, const float* centroids,
                                 const float* codebooks, const float* list_means,
                                 hipStream_t stream) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!seq_lens || !list_ids || !codes || !norms || !centroids || !codebooks || !list_means)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "every index argument must be non-NULL");
    pqhsa_status st = check_device(c);
    if (st != PQHSA_OK) return st;
    const Dims& D = c->D;
    const int B = D.B, Hkv = D.Hkv, L = D.n_list;
    const size_t rc = D.rcap;
    std::vector<int32_t> lens(seq_lens, seq_lens + B);
    for (int b = 0; b < B; ++b)
        if (lens[b] < D.n_sink + D.n_local || lens[b] > D.rcap)
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT,
                        "seq_lens[%d] = %d outside [n_sink + n_local, max_seq] = [%d, %d]", b, lens[b],
                        D.n_sink + D.n_local, D.rcap);
    c->prepared = false;

    const size_t BG = static_cast<size_t>(B) * Hkv;
    hipError_t e = hipMemcpyAsync(c->ids_tm, list_ids, BG * rc * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->codes_tm, codes, BG * rc * c->shape.pq_m, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(c->norms_tm, norms, BG * rc * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->centroids, centroids, BG * L * kHeadDim * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->codebooks, codebooks, BG * c->codebook_floats * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->means, list_means, BG * L * kHeadDim * 4, hipMemcpyDeviceToDevice, stream);
    if (e != hipSuccess) return hip_fail(c, e, "copying the index");
    return relayout(c, lens, stream);
}

pqhsa_status pqhsa_index_update(pqhsa_ctx* c, const int32_t* new_seq_lens, const void* k_cache,
                                const void* v_cache, const int64_t* kv_strides, hipStream_t stream) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!c->prepared) return fail(c, PQHSA_ERR_NOT_PREPARED, "pqhsa_index_prepare has not succeeded");
    if (!new_seq_lens || !k_cache || !v_cache || !kv_strides)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "new_seq_lens, k_cache, v_cache and kv_strides must be non-NULL");
    pqhsa_status st = check_device(c);
    if (st != PQHSA_OK) return st;
    KV kv;
    // the update reads no query and writes no output: the cache stands in for both
    st = check_kv(c, k_cache, k_cache, v_cache, kv_strides, k_cache, &kv);
    if (st != PQHSA_OK) return st;
    const Dims& D = c->D;
    std::vector<int32_t> lens(new_seq_lens, new_seq_lens + D.B);
    BatchInts lo{}, hi{};
    int max_new = 0;
    for (int b = 0; b < D.B; ++b) {
        if (lens[b] < c->cur_len[b] || lens[b] > D.rcap)
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT,
                        "new_seq_lens[%d] = %d outside [current N_b, max_seq] = [%d, %d]", b, lens[b],
                        c->cur_len[b], D.rcap);
        lo.v[b] = c->seq_lens[b] - D.n_local;   // the current end of R_b
        hi.v[b] = lens[b] - D.n_local;
        max_new = std::max(max_new, hi.v[b] - lo.v[b]);
    }
    // encode, merge the new tokens into the other half of the list-major
    // arrays and refresh the means, swap the halves, then gather codes and
    // norms into the new order
    c->prepared = false;
    hipError_t e = launch_encode_update(D, lo, hi, max_new, kv, c->centroids, c->codebooks,
                                        c->ids_tm, c->codes_tm, c->norms_tm, stream);
    if (e == hipSuccess)
        e = launch_update_lists(D, lo, hi, kv, c->ids_tm, c->loff, c->perm, c->pos_word,
                                c->loff_alt, c->shift, c->perm_alt, c->pos_alt, c->n_r_dev, c->n_seq_dev, c->means, c->mean_sums, stream);
    if (e != hipSuccess) return hip_fail(c, e, "launching the index update");
    std::swap(c->perm, c->perm_alt);
    std::swap(c->pos_word, c->pos_alt);
    std::swap(c->loff, c->loff_alt);
    e = launch_prepare_gather(D, c->codes_tm, c->norms_tm, c->index(), c->codes, c->norms, stream);
    if (e == hipSuccess)
        e = launch_sample_slab(D, c->index(), c->samp_codes, c->samp_norms, c->samp_list, stream);
    if (e == hipSuccess) e = launch_glob_mean(D, c->index(), c->glob_mean, stream);
    if (e != hipSuccess) return hip_fail(c, e, "launching the index rebuild");
    int nr_max = 0;
    for (int b = 0; b < D.B; ++b) {
        c->n_r[b] = lens[b] - D.n_sink - D.n_local;
        nr_max = std::max(nr_max, c->n_r[b]);
    }
    c->seq_lens = lens;
    c->cur_len = lens;
    c->scan_nwg = (nr_max + kScanWaves * kSub - 1) / (kScanWaves * kSub);
    c->prepared = true;
    return PQHSA_OK;
}

pqhsa_status pqhsa_index_build(pqhsa_ctx* c, const int32_t* seq_lens, const void* k_cache,
                               const void* v_cache, const int64_t* kv_strides,
                               const int32_t* init_coarse, const int32_t* init_pq,
                               int32_t n_iter_coarse, int32_t n_iter_pq, hipStream_t stream) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!seq_lens || !k_cache || !v_cache || !kv_strides || !init_coarse || !init_pq)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "every build argument must be non-NULL");
    if (n_iter_coarse < 0 || n_iter_coarse > 64 || n_iter_pq < 0 || n_iter_pq > 64)
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "iteration counts must lie in [0, 64]");
    pqhsa_status st = check_device(c);
    if (st != PQHSA_OK) return st;
    KV kv;
    st = check_kv(c, k_cache, k_cache, v_cache, kv_strides, k_cache, &kv);
    if (st != PQHSA_OK) return st;
    const Dims& D = c->D;
    const size_t rc = D.rcap, BG = static_cast<size_t>(D.B) * D.Hkv, L = D.n_list;
    const int M = c->shape.pq_m, Kc = c->shape.pq_ksub;
    std::vector<int32_t> lens(seq_lens, seq_lens + D.B);
    BatchInts lo{}, hi{};
    int max_n = 0;
    for (int b = 0; b < D.B; ++b) {
        if (lens[b] < D.n_sink + D.n_local || lens[b] > D.rcap)
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT,
                        "seq_lens[%d] = %d outside [n_sink + n_local, max_seq] = [%d, %d]", b, lens[b],
                        D.n_sink + D.n_local, D.rcap);
        lo.v[b] = D.n_sink;
        hi.v[b] = lens[b] - D.n_local;
        max_n = std::max(max_n, hi.v[b] - lo.v[b]);
    }
    // the drawn starting tokens must lie in R_b
    std::vector<int32_t> ic(BG * L), ip(BG * M * Kc);
    hipError_t e = hipMemcpyAsync(ic.data(), init_coarse, ic.size() * 4, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(ip.data(), init_pq, ip.size() * 4, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(c, e, "copying the starting tokens to the host");
    for (size_t i = 0; i < ic.size() + ip.size(); ++i) {
        const bool coarse = i < ic.size();
        const size_t bg = coarse ? i / L : (i - ic.size()) / (static_cast<size_t>(M) * Kc);
        const int t = coarse ? ic[i] : ip[i - ic.size()];
        const int b = static_cast<int>(bg / D.Hkv);
        if (t < lo.v[b] || t >= hi.v[b])
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "%s starting token %d of (b %d, kv head %d) outside R_b",
                        coarse ? "coarse" : "subspace", t, b, static_cast<int>(bg % D.Hkv));
    }
    c->prepared = false;
    BuildBufs bb{};
    const size_t n_offs = std::max(BG * (L + 1), BG * M * (Kc + 1));
    e = hipMalloc(&bb.order, BG * M * rc * 4);
    if (e == hipSuccess) e = hipMalloc(&bb.offs, n_offs * 4);
    if (e == hipSuccess) e = hipMalloc(&bb.dist_c, BG * rc * 4);
    if (e == hipSuccess) e = hipMalloc(&bb.dist_f, BG * rc * M * 4);
    {
        // the grouping's per-segment counts: problems x segments x keys
        int max_r = 0;
        for (int b = 0; b < D.B; ++b) max_r = std::max(max_r, hi.v[b] - lo.v[b]);
        const size_t nseg = (static_cast<size_t>(max_r) + kBuildSegTok - 1) / kBuildSegTok;
        const size_t n_hist = std::max<size_t>(1, nseg * std::max(BG * L, BG * M * Kc));
        if (e == hipSuccess) e = hipMalloc(&bb.seg_hist, n_hist * 4);
    }
    auto release = [&]() {
        hipFree(bb.order);
        hipFree(bb.offs);
        hipFree(bb.dist_c);
        hipFree(bb.dist_f);
        hipFree(bb.seg_hist);
    };
    if (e != hipSuccess) {
        release();
        return hip_fail(c, e, "allocating the build scratch");
    }
    float* C = c->centroids;
    float* P = c->codebooks;
    if (e == hipSuccess) e = hipMemsetAsync(C, 0, BG * L * kHeadDim * 4, stream);
    if (e == hipSuccess) e = hipMemsetAsync(P, 0, BG * c->codebook_floats * 4, stream);
    // keep_lists: the subspace passes reuse the final lists instead of
    // searching the (unchanged) centroids again
    // an assignment pass on the matrix cores: the coarse search (unless the
    // lists are kept), then the codeword search of every subspace, which
    // also writes the norms
    auto encode = [&](int keep_lists) {
        if (e == hipSuccess && !keep_lists)
            e = launch_assign(D, lo, hi, max_n, kv, C, c->ids_tm, bb.dist_c, stream);
        if (e == hipSuccess)
            e = launch_subspace(D, lo, hi, max_n, kv, C, P, c->ids_tm, c->codes_tm, c->norms_tm,
                                bb.dist_f, stream);
    };
    if (e == hipSuccess) e = hipMemsetAsync(c->ids_tm, 0, BG * rc * 4, stream);
    encode(1);   // the norms of R (codes against the zero model are discarded)
    if (e == hipSuccess) e = launch_init_centers(D, 0, kv, init_coarse, c->ids_tm, c->norms_tm, C, C, stream);
    for (int it = 0; it < n_iter_coarse; ++it) {
        encode(0);
        if (e == hipSuccess) e = launch_group(D, lo, hi, 0, c->ids_tm, c->codes_tm, bb, stream);
        if (e == hipSuccess) e = launch_centers(D, lo, hi, 0, kv, c->ids_tm, c->norms_tm, C, bb, C, stream);
        if (e == hipSuccess) e = launch_reseed(D, lo, hi, 0, kv, c->ids_tm, c->norms_tm, C, bb, C, stream);
    }
    encode(0);   // the final lists
    if (e == hipSuccess) e = launch_init_centers(D, 1, kv, init_pq, c->ids_tm, c->norms_tm, C, P, stream);
    for (int it = 0; it < n_iter_pq; ++it) {
        encode(1);
        if (e == hipSuccess) e = launch_group(D, lo, hi, 1, c->ids_tm, c->codes_tm, bb, stream);
        if (e == hipSuccess) e = launch_centers(D, lo, hi, 1, kv, c->ids_tm, c->norms_tm, C, bb, P, stream);
        if (e == hipSuccess) e = launch_reseed(D, lo, hi, 1, kv, c->ids_tm, c->norms_tm, C, bb, P, stream);
    }
    encode(1);   // the final codes
    if (e == hipSuccess) e = launch_group(D, lo, hi, 0, c->ids_tm, c->codes_tm, bb, stream);
    if (e == hipSuccess)
        e = launch_centers(D, lo, hi, 2, kv, c->ids_tm, c->norms_tm, C, bb, c->means, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    release();
    if (e != hipSuccess) return hip_fail(c, e, "building the index");
    return relayout(c, lens, stream);
}

pqhsa_status pqhsa_set_lengths(pqhsa_ctx* c, const int32_t* seq_lens) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!c->prepared) return fail(c, PQHSA_ERR_NOT_PREPARED, "pqhsa_index_prepare has not succeeded");
    if (!seq_lens) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "seq_lens is NULL");
    for (int b = 0; b < c->D.B; ++b) {
        const int lo = c->seq_lens[b];
        const int hi = std::min(lo + kTailGrowth, c->D.rcap);
        if (seq_lens[b] < lo || seq_lens[b] > hi)
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT,
                        "seq_lens[%d] = %d outside [indexed N_b, indexed N_b + %d] = [%d, %d]", b,
                        seq_lens[b], kTailGrowth, lo, hi);
    }
    c->cur_len.assign(seq_lens, seq_lens + c->D.B);
    return PQHSA_OK;
}

pqhsa_status pqhsa_index_export_tokens(pqhsa_ctx* c, int32_t* list_ids, uint8_t* codes,
                                       float* norms, float* list_means, float* centroids,
                                       float* codebooks, hipStream_t stream) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!c->prepared) return fail(c, PQHSA_ERR_NOT_PREPARED, "pqhsa_index_prepare has not succeeded");
    pqhsa_status st = check_device(c);
    if (st != PQHSA_OK) return st;
    const size_t BGR = static_cast<size_t>(c->D.B) * c->D.Hkv * c->D.rcap;
    const size_t nmean = static_cast<size_t>(c->D.B) * c->D.Hkv * c->D.n_list * kHeadDim;
    hipError_t e = hipSuccess;
    auto D2D = [&](void* dst, const void* src, size_t bytes) {
        if (dst && e == hipSuccess) e = hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, stream);
    };
    D2D(list_ids, c->ids_tm, BGR * 4);
    D2D(codes, c->codes_tm, BGR * c->shape.pq_m);
    D2D(norms, c->norms_tm, BGR * 4);
    D2D(list_means, c->means, nmean * 4);
    D2D(centroids, c->centroids, nmean * 4);
    D2D(codebooks, c->codebooks,
        static_cast<size_t>(c->D.B) * c->D.Hkv * c->codebook_floats * 4);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(c, e, "exporting the index");
    return PQHSA_OK;
}

// block_table null: contiguous cache; else paged (see check_pages)
// The decode call. With dev_lens / dev_topk (device arrays) the budgets and
// lengths are read on the device by the call's first kernel instead of being
// checked and passed by value; then no stage timing is recorded.
static pqhsa_status decode_impl(pqhsa_ctx* c, const void* q, const void* k, const void* v,
                                const int64_t* strides, const int32_t* block_table,
                                int32_t max_blocks, int32_t page_size, const int32_t* topk,
                                float* out, hipStream_t stream, BatchArgs* ba_out,
                                const int32_t* dev_lens = nullptr, const int32_t* dev_topk = nullptr) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!c->prepared) return fail(c, PQHSA_ERR_NOT_PREPARED, "pqhsa_index_prepare has not succeeded");
    KV kv;
    pqhsa_status st = check_kv(c, q, k, v, strides, out, &kv);
    if (st != PQHSA_OK) return st;
    if (block_table) {
        st = check_pages(c, block_table, max_blocks, page_size, &kv);
        if (st != PQHSA_OK) return st;
    }
    const bool dev_args = dev_topk != nullptr;
    if (!topk && !dev_args) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "topk is NULL");
    st = check_device(c);
    if (st != PQHSA_OK) return st;
    const Dims& D = c->D;
    BatchArgs ba{};
    int nsplit = 1;   // exact-set splits this call needs per row
    Work w = c->w;
    if (dev_args) {
        // every split the partial buffer holds: surplus workgroups exit
        for (int b = 0; b < D.B; ++b) ba.n_r[b] = c->n_r[b];
        nsplit = c->nsplit_max;
        w.ba_dev = c->ba_dev;
        w.dev_lens = dev_lens;
        w.dev_topk = dev_topk;
    }
    for (int b = 0; b < D.B && !dev_args; ++b) {
        if (topk[b] < 0 || topk[b] > c->n_r[b] || topk[b] > c->shape.max_topk)
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "topk[%d] = %d outside [0, min(|R_b| = %d, max_topk = %d)]",
                        b, topk[b], c->n_r[b], c->shape.max_topk);
        ba.topk[b] = topk[b];
        ba.n_r[b] = c->n_r[b];
        ba.n_tail[b] = c->cur_len[b] - D.n_sink - c->n_r[b];
        nsplit = std::max(nsplit, (D.n_sink + ba.n_tail[b] + topk[b] + D.attn_rows - 1) / D.attn_rows);
    }
    const Index ix = c->index();
    const bool timed = c->timing != 0 && !dev_args;
    hipError_t e = hipSuccess;
    if (timed && !c->events_made) {
        for (auto& ev : c->ev)
            if (e == hipSuccess) e = hipEventCreate(&ev);
        if (e != hipSuccess) return hip_fail(c, e, "hipEventCreate");
        c->events_made = true;
    }
    c->timed_valid = false;
    // with stage timing, each kernel records events around its own execution
    auto tm = [&](int i) {
        return timed ? KTiming{c->ev[2 * i], c->ev[2 * i + 1]} : KTiming{};
    };
    if (e == hipSuccess) e = launch_prologue(D, ba, kv, ix, w, c->bias, stream, tm(0));
    if (e == hipSuccess) e = launch_scan(D, ba, ix, w, c->scan_nwg, stream, tm(1));
    if (e == hipSuccess)
        e = launch_select(D, ba, ix, w, c->force_fallback, c->variant == PQHSA_VARIANT_BX, stream, tm(2));
    if (e == hipSuccess)
        e = launch_attend(D, ba, kv, ix, w, nsplit, c->nsplit_max, c->variant, stream, tm(3));
    if (e == hipSuccess) e = launch_merge(D, ba, w, out, c->nsplit_max, c->variant, stream, tm(4));
    if (e != hipSuccess) return hip_fail(c, e, "enqueueing the decode kernels");
    c->timed_valid = timed;
    if (ba_out) *ba_out = ba;
    return PQHSA_OK;
}

pqhsa_status pqhsa_decode(pqhsa_ctx* c, const void* q, const void* k, const void* v,
                          const int64_t* kv_strides, const int32_t* topk, float* out,
                          hipStream_t stream) {
    return decode_impl(c, q, k, v, kv_strides, nullptr, 0, 0, topk, out, stream, nullptr);
}

pqhsa_status pqhsa_decode_device_args(pqhsa_ctx* c, const void* q, const void* k, const void* v,
                                      const int64_t* kv_strides, const int32_t* seq_lens,
                                      const int32_t* topk, float* out, hipStream_t stream) {
    if (c && (!seq_lens || !topk))
        return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "seq_lens and topk must be non-NULL device arrays");
    return decode_impl(c, q, k, v, kv_strides, nullptr, 0, 0, nullptr, out, stream, nullptr, seq_lens,
                       topk);
}

pqhsa_status pqhsa_decode_paged(pqhsa_ctx* c, const void* q, const void* k_pages,
                                const void* v_pages, const int64_t* page_strides,
                                const int32_t* block_table, int32_t max_blocks, int32_t page_size,
                                const int32_t* topk, float* out, hipStream_t stream) {
    if (c && !block_table) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "block_table is NULL");
    return decode_impl(c, q, k_pages, v_pages, page_strides, block_table, max_blocks, page_size,
                       topk, out, stream, nullptr);
}

pqhsa_status pqhsa_decode_debug(pqhsa_ctx* c, const void* q, const void* k, const void* v,
                                const int64_t* kv_strides, const int32_t* topk, float* out,
                                int32_t* selected, int32_t* unselected_per_list, float* scores,
                                hipStream_t stream) {
    if (c && (selected || unselected_per_list) && topk) {
        for (int b = 0; b < c->D.B; ++b)
            if (topk[b] > 8192)
                return fail(c, PQHSA_ERR_UNSUPPORTED, "the debug call sorts at most 8192 selected tokens per row");
    }
    BatchArgs ba{};
    pqhsa_status st = decode_impl(c, q, k, v, kv_strides, nullptr, 0, 0, topk, out, stream, &ba);
    if (st != PQHSA_OK) return st;
    hipError_t e = launch_debug(c->D, ba, c->index(), c->w, selected, unselected_per_list, scores, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(c, e, "running the debug kernels");
    return PQHSA_OK;
}

pqhsa_status pqhsa_dense_decode(pqhsa_ctx* c, const void* q, const void* k, const void* v,
                                const int64_t* kv_strides, const int32_t* seq_lens, float* out,
                                hipStream_t stream) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    KV kv;
    pqhsa_status st = check_kv(c, q, k, v, kv_strides, out, &kv);
    if (st != PQHSA_OK) return st;
    if (!seq_lens) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "seq_lens is NULL");
    st = check_device(c);
    if (st != PQHSA_OK) return st;
    BatchInts lens;
    for (int b = 0; b < c->D.B; ++b) {
        if (seq_lens[b] < 1 || seq_lens[b] > c->D.rcap)
            return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "seq_lens[%d] = %d outside [1, max_seq]", b, seq_lens[b]);
        lens.v[b] = seq_lens[b];
    }
    hipError_t e = launch_dense(c->D, kv, lens, c->dense_partial, out, c->dense_nsplit, stream);
    if (e != hipSuccess) return hip_fail(c, e, "enqueueing the dense decode kernels");
    return PQHSA_OK;
}

pqhsa_status pqhsa_dense_decode_noalloc(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                        int32_t head_dim, int32_t kv_dtype, const void* q,
                                        const void* k, const void* v, const int64_t* kv_strides,
                                        const int32_t* seq_lens, float* out, hipStream_t stream) {
    g_create_error.clear();
    // every check on the host first: nothing below touches the device until
    // the call is known to fit the scratch array
    if (batch < 1 || n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads)
        return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT,
                    "need batch, n_q_heads, n_kv_heads >= 1 and n_kv_heads dividing n_q_heads");
    const int G = n_q_heads / n_kv_heads;
    if (G != 1 && G != 2 && G != 4 && G != 8)
        return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "GQA group size must be 1, 2, 4 or 8");
    if (head_dim != kHeadDim) return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "head_dim must be 128");
    if (kv_dtype != PQHSA_F32 && kv_dtype != PQHSA_BF16)
        return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "kv_dtype must be PQHSA_F32 or PQHSA_BF16");
    if (batch > kMaxBatch) return fail(nullptr, PQHSA_ERR_UNSUPPORTED, "batch must be <= 256");
    KV kv;
    pqhsa_status st = check_kv_dtype(nullptr, kv_dtype, q, k, v, kv_strides, out, &kv);
    if (st != PQHSA_OK) return st;
    if (!seq_lens) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "seq_lens is NULL");
    BatchInts lens;
    int n_max = 0;
    for (int b = 0; b < batch; ++b) {
        if (seq_lens[b] < 1 || seq_lens[b] > kMaxSeq)
            return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "seq_lens[%d] = %d outside [1, 2^20]", b,
                        seq_lens[b]);
        lens.v[b] = seq_lens[b];
        n_max = std::max(n_max, seq_lens[b]);
    }
    // the split partials of every row, in the fixed scratch array
    const int nsplit = (n_max + kDenseRows - 1) / kDenseRows;
    const size_t need = static_cast<size_t>(batch) * n_q_heads * nsplit * kPartStride * sizeof(float);
    if (need > static_scratch_bytes())
        return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT,
                    "batch %d x %d query heads x %d splits of %d tokens need %zu bytes of scratch; "
                    "the fixed scratch holds %zu",
                    batch, n_q_heads, nsplit, kDenseRows, need, static_scratch_bytes());
    void* scratch = nullptr;
    hipError_t e = static_scratch(&scratch);
    if (e != hipSuccess) return fail(nullptr, PQHSA_ERR_HIP, "scratch address: %s", hipGetErrorString(e));
    Dims D{};
    D.B = batch;
    D.Hq = n_q_heads;
    D.Hkv = n_kv_heads;
    D.G = G;
    D.inv_sqrt_d = static_cast<float>(1.0 / std::sqrt(static_cast<double>(kHeadDim)));
    e = launch_dense(D, kv, lens, static_cast<float*>(scratch), out, nsplit, stream);
    if (e != hipSuccess)
        return fail(nullptr, PQHSA_ERR_HIP, "enqueueing the dense decode kernels: %s", hipGetErrorString(e));
    return PQHSA_OK;
}

pqhsa_status pqhsa_index_export(pqhsa_ctx* c, int32_t* perm, int32_t* offsets, hipStream_t stream) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    c->err.clear();
    if (!c->prepared) return fail(c, PQHSA_ERR_NOT_PREPARED, "pqhsa_index_prepare has not succeeded");
    const size_t BG = static_cast<size_t>(c->D.B) * c->D.Hkv;
    hipError_t e = hipSuccess;
    if (perm) e = hipMemcpyAsync(perm, c->perm, BG * c->D.rcap * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess && offsets)
        e = hipMemcpyAsync(offsets, c->loff, BG * (c->D.n_list + 1) * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(c, e, "exporting the index");
    return PQHSA_OK;
}

pqhsa_status pqhsa_set_option(pqhsa_ctx* c, int32_t option, int64_t value) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    switch (option) {
        case PQHSA_OPT_FORCE_FALLBACK: c->force_fallback = value != 0; return PQHSA_OK;
        case PQHSA_OPT_STAGE_TIMING: c->timing = value != 0; return PQHSA_OK;
        case PQHSA_OPT_THRESHOLD_BIAS: c->bias = static_cast<float>(value) / 1000.0f; return PQHSA_OK;
        case PQHSA_OPT_VARIANT:
            if (value != PQHSA_VARIANT_B && value != PQHSA_VARIANT_T && value != PQHSA_VARIANT_C &&
                value != PQHSA_VARIANT_BX)
                return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "variant %lld is not one of B, T, C, Bx",
                            static_cast<long long>(value));
            c->variant = static_cast<int>(value);
            return PQHSA_OK;
        default: return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "unknown option %d", option);
    }
}

pqhsa_status pqhsa_stage_times(pqhsa_ctx* c, float* ms, int32_t n, int32_t* n_out) {
    if (!c) return fail(nullptr, PQHSA_ERR_INVALID_ARGUMENT, "ctx is NULL");
    if (!ms || !n_out) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "ms and n_out must be non-NULL");
    if (!c->timed_valid) return fail(c, PQHSA_ERR_INVALID_ARGUMENT, "no decode call was timed");
    hipError_t e = hipEventSynchronize(c->ev[2 * kStages - 1]);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize");
    for (int i = 0; i < kStages && i < n; ++i) {
        float t = 0.0f;
        e = hipEventElapsedTime(&t, c->ev[2 * i], c->ev[2 * i + 1]);
        if (e != hipSuccess) return hip_fail(c, e, "hipEventElapsedTime");
        ms[i] = t;
    }
    *n_out = kStages;
    return PQHSA_OK;
}

}  // extern "C"
