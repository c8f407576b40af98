// Host side of the engine: the C ABI of include/warp.h, argument validation,
// device memory of the index and of the per-search scratch, and the launch
// sequence of one search (Section 4: candidate generation, decompression,
// scoring). Queries are processed in waves; a wave holds one token-max table
// row per query token and one sort key per document for each of its queries.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_set>
#include <utility>
#include <vector>

#include "engine.h"
#include "warp.h"

using namespace warp;

// Scratch of warp_search_noalloc: one array per GPU (each device holds its own copy), kept
// until the process ends. Host code never uses this name as an address: the device address
// comes from hipGetSymbolAddress, once per device, when the first index is loaded on it.
constexpr size_t kNoAllocBytes = (size_t)256 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

#define HIP_TRY(expr)                                                                         \
    do {                                                                                      \
        hipError_t e_ = (expr);                                                               \
        if (e_ != hipSuccess) return fail(WARP_EDEVICE, "%s failed: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

constexpr int kStages = 6;

struct DevBuf {
    void* p = nullptr;
    size_t bytes = 0;
};

}  // namespace

struct warp_index {
    int device = 0;
    int32_t n_c = 0, n_docs = 0, nbits = 0;
    int64_t n_emb = 0;
    float* centroids = nullptr;
    int64_t* offsets = nullptr;
    int32_t* sizes = nullptr;
    int32_t* chunk_c = nullptr;  // the index's chunks in a fixed pseudo-random order (see WaveArgs)
    int32_t* chunk_k = nullptr;
    int64_t n_chunks = 0;
    int32_t* doc_ids = nullptr;
    uint8_t* codes = nullptr;
    float* weights = nullptr;
    int32_t* err = nullptr;
    hipStream_t stream = nullptr;
    int scan_grid = 0;     // persistent workgroups of the residual scan
    int narrow_grid = 0;   // workgroups of the narrow scan (four waves, one chunk per wave at a time)
    int n_cu = 0;          // compute units of the device
    // per-search scratch, grown on demand
    DevBuf filter, sel, base, seg_pref, m_fixed, tokmax, keys, qpart;
    // Token-max table [wave query slot][token][document]. The rows of query slot q carry an
    // epoch e_q >= 1 that every wave using the slot advances: its cells hold
    // t + e_q 2^w + 2^(w-1), where 2^(w-1) exceeds every |t| that the bucket weights and the
    // norm limits allow, so values of earlier epochs lie below e_q 2^w, the fold reads them as
    // absent and never resets a cell. A slot's rows are zeroed before a wave would take it
    // past the last epoch, 2^(32-w) - 1. When no bit is spare and in the Eq.-1-literal mode,
    // a cell holds t + 2^31, 0 is absent, and the fold resets every cell it reads.
    int32_t tab_w = 32;
    int32_t tab_epochs = 0;        // 2^(32-w) - 1, if at least 2; 0: the fold resets cells
    int64_t tab_cells = 0;         // cells the table holds
    int32_t tab_T = 0;             // tokens per query slot of the epochs' layout
    bool tab_force_zero = false;   // zero every slot first (after a query-norm error)
    std::vector<uint32_t> slot_ep; // epoch of each query slot's rows; 0: all zero
    DevBuf q_epoch;                // device copy of slot_ep
    DevBuf ccount, cursor, pair_start, coff, plist, qdig;
    DevBuf list_rec, list_item, cblk;  // the wave's probed chunks (see WaveArgs)
    DevBuf list_rec2;                  // the wave's probed chunks of the narrow scan
    DevBuf scan_queue;
    DevBuf full_sel, full_topk;  // sort scratch of the sorting selection and of k > kMaxK
    DevBuf sel_hist, sel_lists, sel_cnt;  // split selection of small waves
    bool force_full_select = false;       // the blocking search's retry after a selection overflow
    int32_t scoring = WARP_SCORING_PAPER;
    DevBuf tokcnt, doc_len;    // Eq.-1-literal scoring only
    int64_t tokcnt_ready = 0;  // leading elements of tokcnt holding 0
    bool doc_len_ready = false;
    size_t scratch_held = 0;  // bytes of per-search scratch (all DevBufs above and below)
    // staging of the host-pointer calls
    DevBuf st_q, st_ids, st_scores, st_fixed, st_counts, st_sel, st_m, st_bitmap, st_scored;
    std::mutex lock;
    // stage timing
    bool timing = false;
    std::vector<hipEvent_t> ev_pool;
    std::vector<hipEvent_t> ev_pending;  // groups of kStages + 1
    double stage_ms[kStages] = {0};
    int64_t stage_launches[kStages] = {0};
};

namespace {

int grow(DevBuf& b, size_t bytes) {
    if (bytes == 0) bytes = 16;
    if (b.bytes >= bytes) return WARP_OK;
    if (b.p) (void)hipFree(b.p);
    b.p = nullptr;
    b.bytes = 0;
    if (hipMalloc(&b.p, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return fail(WARP_ENOMEM, "hipMalloc of %zu bytes failed", bytes);
    }
    b.bytes = bytes;
    return WARP_OK;
}

void release(DevBuf& b) {
    if (b.p) (void)hipFree(b.p);
    b.p = nullptr;
    b.bytes = 0;
}

// Cap on an index's per-search scratch: WARP_MAX_SCRATCH_BYTES if set (bytes), else none.
// A search whose scratch would exceed it fails with WARP_ENOMEM, as if the device memory
// had run out; the waves of a search are sized to stay below it.
size_t scratch_cap() {
    const char* s = std::getenv("WARP_MAX_SCRATCH_BYTES");
    if (!s || !*s) return SIZE_MAX;
    const long long v = std::atoll(s);
    return v < 0 ? 0 : (size_t)v;
}

// grow() for the index's per-search scratch, counted against scratch_cap().
int grow_scratch(warp_index* idx, DevBuf& b, size_t bytes) {
    if (bytes == 0) bytes = 16;
    if (b.bytes >= bytes) return WARP_OK;
    const size_t cap = scratch_cap();
    const size_t after = idx->scratch_held - b.bytes + bytes;
    if (after > cap)
        return fail(WARP_ENOMEM, "search scratch of %zu bytes exceeds WARP_MAX_SCRATCH_BYTES = %zu", after, cap);
    idx->scratch_held -= b.bytes;
    const int rc = grow(b, bytes);
    idx->scratch_held += b.bytes;
    return rc;
}

// Live index handles: a call on a handle that was never returned by a load, or was freed,
// fails with WARP_EINVAL instead of touching freed memory.
std::mutex g_live_lock;
std::unordered_set<const warp_index*>& live_handles() {
    static std::unordered_set<const warp_index*>* s = new std::unordered_set<const warp_index*>();
    return *s;
}

int check_device() {
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n < 1) {
        (void)hipGetLastError();
        return fail(WARP_EDEVICE, "no HIP device is available");
    }
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, dev));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(WARP_EDEVICE, "device %d is %s; this library is built for gfx950 only", dev,
                    prop.gcnArchName);
    return WARP_OK;
}

// Per-device address of `scratch`, set by bind_noalloc_scratch.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_lock;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// Look up this device's copy of `scratch` (device `dev` must be current); once per device.
int bind_noalloc_scratch(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return fail(WARP_EDEVICE, "device %d is out of range", dev);
    std::lock_guard<std::mutex> g(g_scratch_lock);
    if (g_scratch_ptr[dev]) return WARP_OK;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
        (void)hipGetLastError();
        return fail(WARP_EDEVICE, "hipGetSymbolAddress of the no-allocation scratch failed: %s",
                    hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = (unsigned char*)p;
    return WARP_OK;
}

unsigned char* noalloc_scratch(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> g(g_scratch_lock);
    return g_scratch_ptr[dev];
}

bool is_index(const warp_index* idx) {
    if (!idx) return false;
    std::lock_guard<std::mutex> g(g_live_lock);
    return live_handles().count(idx) != 0;
}

// Free everything an index owns (registered or not).
void destroy_index(warp_index* idx) {
    {
        std::lock_guard<std::mutex> g(idx->lock);
        (void)hipSetDevice(idx->device);
        if (idx->stream) (void)hipStreamSynchronize(idx->stream);
        for (void* p : {(void*)idx->centroids, (void*)idx->offsets, (void*)idx->sizes, (void*)idx->chunk_c,
                        (void*)idx->chunk_k, (void*)idx->doc_ids, (void*)idx->codes, (void*)idx->weights,
                        (void*)idx->err})
            if (p) (void)hipFree(p);
        for (DevBuf* b : {&idx->filter, &idx->sel, &idx->base, &idx->seg_pref, &idx->m_fixed, &idx->tokmax,
                          &idx->q_epoch, &idx->tokcnt, &idx->doc_len, &idx->keys, &idx->qpart, &idx->ccount,
                          &idx->cursor, &idx->pair_start, &idx->coff, &idx->plist, &idx->qdig, &idx->list_rec,
                          &idx->list_item, &idx->cblk, &idx->list_rec2, &idx->scan_queue, &idx->full_sel,
                          &idx->full_topk, &idx->sel_hist, &idx->sel_lists, &idx->sel_cnt, &idx->st_q,
                          &idx->st_ids,
                          &idx->st_scores, &idx->st_fixed, &idx->st_counts, &idx->st_sel, &idx->st_m,
                          &idx->st_bitmap, &idx->st_scored})
            release(*b);
        for (hipEvent_t e : idx->ev_pool) (void)hipEventDestroy(e);
        for (hipEvent_t e : idx->ev_pending) (void)hipEventDestroy(e);
        if (idx->stream) (void)hipStreamDestroy(idx->stream);
    }
    delete idx;
}

// Host-side checks of the small index arrays.
int validate_index_host(const float* C, int32_t n_c, int32_t dim, const int64_t* off, int32_t nbits,
                        const float* w, int32_t n_docs) {
    if (n_c < 1) return fail(WARP_EINVAL, "n_centroids must be >= 1 (got %d)", n_c);
    if (dim != kDim) return fail(WARP_ENOTSUP, "dim must be 128 (got %d)", dim);
    if (nbits != 1 && nbits != 2 && nbits != 4 && nbits != 8)
        return fail(WARP_EINVAL, "nbits must be 1, 2, 4 or 8 (got %d)", nbits);
    if (n_docs < 1 || n_docs > kMaxDocs) return fail(WARP_EINVAL, "n_docs must be in [1, 2^24] (got %d)", n_docs);
    if (!C || !off || !w) return fail(WARP_EINVAL, "null index array");
    if (off[0] != 0) return fail(WARP_EINVAL, "cluster_offsets[0] must be 0");
    for (int32_t c = 0; c < n_c; ++c) {
        const int64_t sz = off[c + 1] - off[c];
        if (sz < 0) return fail(WARP_EINVAL, "cluster_offsets decrease at cluster %d", c);
        if (sz > INT32_MAX) return fail(WARP_ENOTSUP, "cluster %d has more than 2^31-1 embeddings", c);
    }
    if (off[n_c] >= (1ll << 40)) return fail(WARP_EINVAL, "more than 2^40 embeddings");
    for (int b = 0; b < (1 << nbits); ++b)
        if (!std::isfinite(w[b]) || std::fabs(w[b]) > kMaxWeight)
            return fail(WARP_EINVAL, "bucket weight %d is not finite or exceeds %.2f in magnitude", b,
                        (double)kMaxWeight);
    for (int32_t c = 0; c < n_c; ++c) {
        double s = 0;
        for (int d = 0; d < kDim; ++d) {
            const float v = C[(int64_t)c * kDim + d];
            if (!std::isfinite(v)) return fail(WARP_EINVAL, "centroid %d is not finite", c);
            s += (double)v * v;
        }
        if (std::fabs(std::sqrt(s) - 1.0) > 1e-3) return fail(WARP_EINVAL, "centroid %d is not of unit norm", c);
    }
    return WARP_OK;
}

// Width w of a token-max cell's value field: the smallest w with 2^(w-1) above a bound B on
// |t| (units of 2^-26) for queries and centroids of norm at most 1 + 1e-3 and these bucket
// weights: |R(S64)| <= 1.001^2 2^26 + 1 and |floor(V 2^-18 + 1/2)| <= (sum_d |Q(q_d)|)
// (max_b |Q(omega_b)|) 2^-18 + 1, with sum_d |Q(q_d)| <= sqrt(128) 1.001 2^22 + 64 and
// |Q(omega_b)| <= |omega_b| 2^22 + 1/2. At the largest weights accepted, w = 32.
int32_t token_value_width(const float* w, int32_t nbits) {
    double wmax = 0;
    for (int b = 0; b < (1 << nbits); ++b) wmax = std::fmax(wmax, std::fabs((double)w[b]));
    const double qsum = std::sqrt((double)kDim) * 1.001 * 4194304.0 + 0.5 * kDim;
    const double bound = 1.001 * 1.001 * 67108864.0 + 1.0 + qsum * (wmax * 4194304.0 + 0.5) / 262144.0 + 1.0;
    const double b = bound * (1.0 + 1e-5) + 64.0;
    int32_t width = 2;
    while (width < 32 && std::ldexp(1.0, width - 1) <= b) ++width;
    return width;
}

int validate_queries_host(const float* q, int64_t n_tok) {
    for (int64_t t = 0; t < n_tok; ++t) {
        double s = 0;
        for (int d = 0; d < kDim; ++d) {
            const float v = q[t * kDim + d];
            if (!std::isfinite(v)) return fail(WARP_EINVAL, "query token %lld is not finite", (long long)t);
            s += (double)v * v;
        }
        if (std::sqrt(s) > 1.0 + 1e-3) return fail(WARP_EINVAL, "query token %lld has norm > 1 + 1e-3", (long long)t);
    }
    return WARP_OK;
}

int validate_search(const warp_index* idx, const void* queries, int32_t n_queries, int32_t n_qtok,
                    int32_t nprobe, int64_t t_prime, int32_t k, const void* ids, const void* scores) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    if (!queries || !ids || !scores) return fail(WARP_EINVAL, "null query or output pointer");
    if (n_queries < 1) return fail(WARP_EINVAL, "n_queries must be >= 1 (got %d)", n_queries);
    if (n_qtok < 1 || n_qtok > kMaxQtok) return fail(WARP_EINVAL, "n_qtok must be in [1, 32] (got %d)", n_qtok);
    if (nprobe < 1 || nprobe > idx->n_c)
        return fail(WARP_EINVAL, "nprobe must be in [1, n_centroids] (got %d)", nprobe);
    if (t_prime < 0) return fail(WARP_EINVAL, "t_prime must be >= 0");
    if (k < 1) return fail(WARP_EINVAL, "k must be >= 1 (got %d)", k);
    return WARP_OK;
}

int finish_load(warp_index* idx, const int64_t* off_host) {
    std::vector<int32_t> sz(idx->n_c);
    for (int32_t c = 0; c < idx->n_c; ++c) sz[c] = (int32_t)(off_host[c + 1] - off_host[c]);
    HIP_TRY(hipMemcpy(idx->sizes, sz.data(), sizeof(int32_t) * idx->n_c, hipMemcpyHostToDevice));
    // the chunks of kMxChunk embeddings of every cluster, shuffled (Fisher-Yates with a fixed
    // xorshift64 stream): the scan's items follow this order
    std::vector<int32_t> cc, ck;
    for (int32_t c = 0; c < idx->n_c; ++c)
        for (int64_t k = 0; k * kMxChunk < sz[c]; ++k) {
            cc.push_back(c);
            ck.push_back((int32_t)k);
        }
    uint64_t x = 0x9E3779B97F4A7C15ull;
    for (int64_t i = (int64_t)cc.size() - 1; i > 0; --i) {
        x ^= x << 13;
        x ^= x >> 7;
        x ^= x << 17;
        const int64_t j = (int64_t)(x % (uint64_t)(i + 1));
        std::swap(cc[i], cc[j]);
        std::swap(ck[i], ck[j]);
    }
    idx->n_chunks = (int64_t)cc.size();
    if (hipMalloc((void**)&idx->chunk_c, cc.size() * 4 + 16) != hipSuccess ||
        hipMalloc((void**)&idx->chunk_k, ck.size() * 4 + 16) != hipSuccess) {
        (void)hipGetLastError();
        return fail(WARP_ENOMEM, "hipMalloc of the index's chunk order failed");
    }
    HIP_TRY(hipMemcpy(idx->chunk_c, cc.data(), cc.size() * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(idx->chunk_k, ck.data(), ck.size() * 4, hipMemcpyHostToDevice));
    launch_fill_i32(idx->err, 1, 0, idx->stream);
    launch_check_docs(idx->doc_ids, idx->n_emb, idx->n_docs, idx->err, idx->stream);
    int32_t err = 0;
    HIP_TRY(hipMemcpyAsync(&err, idx->err, sizeof err, hipMemcpyDeviceToHost, idx->stream));
    HIP_TRY(hipStreamSynchronize(idx->stream));
    if (err & kErrDocRange) return fail(WARP_EINVAL, "a document id is outside [0, n_docs)");
    int cus = 0;
    HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, idx->device));
    idx->scan_grid = cus * scan_mx_blocks_per_cu(idx->nbits);
    idx->n_cu = cus;
    idx->narrow_grid = cus * scan_narrow_blocks_per_cu(idx->nbits);
    return WARP_OK;
}

int load_common(const float* C, int32_t n_c, int32_t dim, const int64_t* off, const int32_t* doc_ids,
                const uint8_t* codes, int32_t nbits, const float* w, int32_t n_docs, warp_index** out,
                bool device_ptrs) {
    if (!out) return fail(WARP_EINVAL, "out is null");
    if (!C || !off || !w || !doc_ids || !codes) return fail(WARP_EINVAL, "null index array");
    if (n_c < 1) return fail(WARP_EINVAL, "n_centroids must be >= 1 (got %d)", n_c);
    if (dim != kDim) return fail(WARP_ENOTSUP, "dim must be 128 (got %d)", dim);
    int rc = WARP_OK;
    if (!device_ptrs) {  // host arrays are checked before any device call
        rc = validate_index_host(C, n_c, dim, off, nbits, w, n_docs);
        if (rc) return rc;
    }
    rc = check_device();
    if (rc) return rc;
    // host copies of the small arrays for validation
    std::vector<float> hC, hw;
    std::vector<int64_t> hoff;
    const float* vC = C;
    const int64_t* voff = off;
    const float* vw = w;
    if (device_ptrs) {
        // the small arrays are read on the host: copy them first, whatever nbits is (an
        // invalid nbits is rejected below before the weights are used)
        if (nbits != 1 && nbits != 2 && nbits != 4 && nbits != 8)
            return fail(WARP_EINVAL, "nbits must be 1, 2, 4 or 8 (got %d)", nbits);
        hC.resize((size_t)n_c * kDim);
        hoff.resize((size_t)n_c + 1);
        hw.resize((size_t)1 << nbits);
        HIP_TRY(hipMemcpy(hC.data(), C, hC.size() * 4, hipMemcpyDeviceToHost));
        HIP_TRY(hipMemcpy(hoff.data(), off, hoff.size() * 8, hipMemcpyDeviceToHost));
        HIP_TRY(hipMemcpy(hw.data(), w, hw.size() * 4, hipMemcpyDeviceToHost));
        vC = hC.data();
        voff = hoff.data();
        vw = hw.data();
    }
    if (device_ptrs) {
        rc = validate_index_host(vC, n_c, dim, voff, nbits, vw, n_docs);
        if (rc) return rc;
    }

    int device = 0;
    HIP_TRY(hipGetDevice(&device));
    rc = bind_noalloc_scratch(device);
    if (rc) return rc;
    warp_index* idx = new warp_index();
    idx->device = device;
    idx->n_c = n_c;
    idx->n_docs = n_docs;
    idx->nbits = nbits;
    idx->n_emb = voff[n_c];
    idx->tab_w = token_value_width(vw, nbits);
    const int32_t epochs = (int32_t)((1ll << (32 - idx->tab_w)) - 1);
    idx->tab_epochs = epochs >= 2 ? epochs : 0;  // one epoch per zeroing saves nothing over resets
    const size_t row = (size_t)kDim * nbits / 8;
    const hipMemcpyKind kind = device_ptrs ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    auto alloc = [&](void** p, size_t bytes) -> int {
        if (hipMalloc(p, bytes ? bytes : 16) != hipSuccess) {
            (void)hipGetLastError();
            return fail(WARP_ENOMEM, "hipMalloc of %zu bytes for the index failed", bytes);
        }
        return WARP_OK;
    };
    rc = alloc((void**)&idx->centroids, (size_t)n_c * kDim * 4);
    if (!rc) rc = alloc((void**)&idx->offsets, ((size_t)n_c + 1) * 8);
    if (!rc) rc = alloc((void**)&idx->sizes, (size_t)n_c * 4);
    if (!rc) rc = alloc((void**)&idx->doc_ids, (size_t)idx->n_emb * 4);
    if (!rc) rc = alloc((void**)&idx->codes, (size_t)idx->n_emb * row + 16);
    if (!rc) rc = alloc((void**)&idx->weights, (size_t)4 << nbits);
    if (!rc) rc = alloc((void**)&idx->err, 64);
    if (!rc && hipStreamCreateWithFlags(&idx->stream, hipStreamNonBlocking) != hipSuccess)
        rc = fail(WARP_EDEVICE, "hipStreamCreate failed");
    if (!rc && (hipMemcpy(idx->centroids, C, (size_t)n_c * kDim * 4, kind) != hipSuccess ||
                hipMemcpy(idx->offsets, off, ((size_t)n_c + 1) * 8, kind) != hipSuccess ||
                hipMemcpy(idx->doc_ids, doc_ids, (size_t)idx->n_emb * 4, kind) != hipSuccess ||
                hipMemcpy(idx->codes, codes, (size_t)idx->n_emb * row, kind) != hipSuccess ||
                hipMemcpy(idx->weights, w, (size_t)4 << nbits, kind) != hipSuccess))
        rc = fail(WARP_EDEVICE, "copying the index to the device failed");
    if (!rc) rc = finish_load(idx, voff);
    if (rc) {
        std::string msg = g_err;
        destroy_index(idx);
        g_err = msg;
        return rc;
    }
    {
        std::lock_guard<std::mutex> g(g_live_lock);
        live_handles().insert(idx);
    }
    *out = idx;
    return WARP_OK;
}

// Zero the rows of every query slot whose epoch is not 0 (runs of consecutive slots at once).
// With `only_last`, only of the slots of the first n at the last epoch, which the next wave
// takes back to epoch 1.
void zero_slots(warp_index* idx, int32_t n, bool only_last, hipStream_t s) {
    const int64_t cells = (int64_t)idx->tab_T * idx->n_docs;
    auto hit = [&](int32_t q) {
        return only_last ? idx->slot_ep[q] == (uint32_t)idx->tab_epochs : idx->slot_ep[q] != 0;
    };
    for (int32_t q = 0; q < n;) {
        if (!hit(q)) {
            ++q;
            continue;
        }
        int32_t q1 = q + 1;
        while (q1 < n && hit(q1)) ++q1;
        launch_zero_cells((uint32_t*)idx->tokmax.p + q * cells, (int64_t)(q1 - q) * cells, s);
        q = q1;
    }
}

void clear_slots(warp_index* idx, hipStream_t s) {
    bool any = false;
    for (uint32_t e : idx->slot_ep) any |= e != 0;
    if (!any) return;
    zero_slots(idx, (int32_t)idx->slot_ep.size(), false, s);
    std::fill(idx->slot_ep.begin(), idx->slot_ep.end(), 0u);
    launch_fill_i32((int32_t*)idx->q_epoch.p, (int64_t)idx->slot_ep.size(), 0, s);
}

// The selection sorts whole score lists (instead of rescoring the boundary bands) for n_probe
// above kMaxProbe, and in the blocking search's retry after a band overflowed.
bool full_select(const warp_index* idx, int32_t P) { return P > kMaxProbe || idx->force_full_select; }

// Workgroups per token of the selection for a wave of n_tok tokens: one for large waves; for
// waves of at most kSplitTokens tokens, enough to give every compute unit three workgroups, with
// at least kSplitSlice centroids each (WARP_SELECT_SLICES sets the number for every wave).
int select_slices(const warp_index* idx, int64_t n_tok) {
    if (const char* e = std::getenv("WARP_SELECT_SLICES")) {
        const long v = std::atol(e);
        return v < 1 ? 1 : (v > 256 ? 256 : (int)v);
    }
    if (n_tok > kSplitTokens || n_tok < 1) return 1;
    int64_t sl = (3 * (int64_t)idx->n_cu + n_tok - 1) / n_tok;
    const int64_t by_size = idx->n_c / kSplitSlice;
    if (sl > by_size) sl = by_size;
    if (sl > 64) sl = 64;
    return sl < 2 ? 1 : (int)sl;
}

// Tokens whose split-selection scratch waves of n_tok tokens reserve: all of them if such a wave
// splits its selection, else none (a smaller last wave of a larger search then keeps one
// workgroup per token).
int64_t split_tokens(const warp_index* idx, int64_t n_tok) {
    return select_slices(idx, n_tok) > 1 ? n_tok : 0;
}

// Device scratch for a wave of `qw` queries of `T` tokens; the fills are enqueued on the
// search stream `s`, after the searches before it.
int reserve(warp_index* idx, int32_t qw, int32_t T, int32_t P, int32_t k, hipStream_t s) {
    const int64_t n_tok = (int64_t)qw * T;
    int rc = WARP_OK;
    if (!rc) rc = grow_scratch(idx, idx->filter, (size_t)n_tok * idx->n_c * 2);
    if (!rc) rc = grow_scratch(idx, idx->sel, (size_t)n_tok * P * 4);
    if (!rc) rc = grow_scratch(idx, idx->base, (size_t)n_tok * P * 4);
    if (!rc) rc = grow_scratch(idx, idx->seg_pref, (size_t)n_tok * (P + 1) * 8);
    if (!rc) rc = grow_scratch(idx, idx->m_fixed, (size_t)n_tok * 8);
    if (!rc) rc = grow_scratch(idx, idx->keys, (size_t)qw * idx->n_docs * 8);
    if (!rc) rc = grow_scratch(idx, idx->qpart, (size_t)qw * (((size_t)idx->n_docs + 255) / 256) * 16);
    if (!rc) rc = grow_scratch(idx, idx->ccount, (size_t)idx->n_c * 4);
    if (!rc) rc = grow_scratch(idx, idx->cursor, (size_t)idx->n_c * 4);
    if (!rc) rc = grow_scratch(idx, idx->pair_start, ((size_t)idx->n_c + 1) * 4);
    if (!rc) rc = grow_scratch(idx, idx->coff, (((size_t)idx->n_c + kPairBlock - 1) / kPairBlock) * 8);
    if (!rc) rc = grow_scratch(idx, idx->plist, (size_t)n_tok * P * 8);
    if (!rc) rc = grow_scratch(idx, idx->qdig, (size_t)n_tok * kQdigBytes);
    const int64_t cblocks = (idx->n_chunks + kPlanBlock - 1) / kPlanBlock;
    if (!rc) rc = grow_scratch(idx, idx->list_rec, (size_t)idx->n_chunks * 16);
    if (!rc) rc = grow_scratch(idx, idx->list_rec2, (size_t)idx->n_chunks * 16);
    if (!rc) rc = grow_scratch(idx, idx->list_item, ((size_t)idx->n_chunks + 3) * 8);  // + the two counts
    if (!rc) rc = grow_scratch(idx, idx->cblk, (size_t)cblocks * 24);
    if (!rc) rc = grow_scratch(idx, idx->scan_queue, 256);
    if (!rc && full_select(idx, P)) rc = grow_scratch(idx, idx->full_sel, select_full_bytes(n_tok, idx->n_c));
    if (!rc && k > kMaxK) rc = grow_scratch(idx, idx->full_topk, topk_full_bytes(idx->n_docs));
    const int64_t st = split_tokens(idx, n_tok);
    if (!rc) rc = grow_scratch(idx, idx->sel_hist, (size_t)st * kSelBins * 8);
    if (!rc) rc = grow_scratch(idx, idx->sel_lists, (size_t)st * 2 * kSelCap * 4);
    if (!rc) rc = grow_scratch(idx, idx->sel_cnt, (size_t)st * 2 * 4);
    if (rc) return rc;
    // the token-max table and its query slots' epochs. All slots are zeroed before a search
    // that resets cells or lays the table out with another token count, and after a search
    // whose queries failed the norm check (their scores can exceed 2^(w-1)).
    const int64_t need = n_tok * idx->n_docs;
    if (idx->tab_cells < need) {
        idx->tab_cells = 0;
        rc = grow_scratch(idx, idx->tokmax, (size_t)need * 4);
        if (rc) return rc;
        launch_zero_cells((uint32_t*)idx->tokmax.p, need, s);
        idx->tab_cells = need;
        std::fill(idx->slot_ep.begin(), idx->slot_ep.end(), 0u);
        if (idx->q_epoch.p) launch_fill_i32((int32_t*)idx->q_epoch.p, (int64_t)idx->slot_ep.size(), 0, s);
    }
    const bool resets = idx->scoring == WARP_SCORING_EQ1_LITERAL || idx->tab_epochs == 0;
    if (idx->tab_force_zero || resets || T != idx->tab_T || (int64_t)idx->slot_ep.size() < qw) {
        clear_slots(idx, s);
        idx->tab_force_zero = false;
        idx->tab_T = T;
    }
    if ((int64_t)idx->slot_ep.size() < qw) {
        rc = grow_scratch(idx, idx->q_epoch, (size_t)qw * 4);
        if (rc) return rc;
        idx->slot_ep.assign((size_t)qw, 0u);
        launch_fill_i32((int32_t*)idx->q_epoch.p, qw, 0, s);
    }
    if (idx->scoring == WARP_SCORING_EQ1_LITERAL) {
        if ((int64_t)(idx->tokcnt.bytes / 4) < need) {
            rc = grow_scratch(idx, idx->tokcnt, (size_t)need * 4);
            if (rc) return rc;
            idx->tokcnt_ready = 0;
        }
        if (!idx->doc_len_ready) {
            rc = grow_scratch(idx, idx->doc_len, (size_t)idx->n_docs * 4);
            if (rc) return rc;
            launch_doc_len(idx->doc_ids, idx->n_emb, (int32_t*)idx->doc_len.p, idx->n_docs, s);
        }
        if (idx->tokcnt_ready < need) launch_fill_i32((int32_t*)idx->tokcnt.p, need, 0, s);
        idx->doc_len_ready = true;
        idx->tokcnt_ready = need;
    }
    return WARP_OK;
}

// Queries per wave: as many as the scratch budget holds. The budget is
// WARP_SCRATCH_MB if set, else 80% of the device memory that is free or already
// held as scratch by this index. A larger wave lets the cluster-major scan read
// each probed cluster once for more queries. The sorting selection sorts the wave's
// n_tok n_c scores, at most 2^31 of them.
int32_t wave_queries(const warp_index* idx, int32_t n_queries, int32_t T, int32_t P) {
    const size_t held = idx->tokmax.bytes + idx->filter.bytes + idx->keys.bytes + idx->plist.bytes +
                        idx->qdig.bytes;
    size_t budget = 0;
    if (const char* s = std::getenv("WARP_SCRATCH_MB")) {
        budget = (size_t)std::atoll(s) << 20;
    } else {
        size_t free_b = 0, total_b = 0;
        if (hipMemGetInfo(&free_b, &total_b) != hipSuccess) {
            (void)hipGetLastError();
            free_b = (size_t)8 << 30;
        }
        budget = (size_t)(0.8 * (double)(free_b + held));
    }
    budget = std::min(budget, scratch_cap());
    const bool full = full_select(idx, P);
    const size_t per = (size_t)T * idx->n_docs * (idx->scoring == WARP_SCORING_EQ1_LITERAL ? 8 : 4) +
                       (size_t)idx->n_docs * 8 + (size_t)T * idx->n_c * 2 + (size_t)T * P * 32 +
                       (size_t)T * 1024 + (full ? select_full_bytes(T, idx->n_c) : 0);
    const int64_t sort_cap = ((int64_t)1 << 31) / ((int64_t)T * idx->n_c);
    auto clamp = [&](int64_t q) {
        if (q > n_queries) q = n_queries;
        if (q > 65535) q = 65535;
        if (full && q > sort_cap) q = sort_cap;
        return q < 1 ? (int64_t)1 : q;
    };
    return (int32_t)clamp((int64_t)(budget / per));
}

// Blocks the top-k may list for its pruned passes: kTopkListCap, or fewer with
// WARP_TOPK_LIST_BLOCKS (0 turns the pruning off).
int32_t topk_list_cap() {
    int64_t v = kTopkListCap;
    if (const char* s = std::getenv("WARP_TOPK_LIST_BLOCKS")) v = std::atoll(s);
    return (int32_t)(v < 0 ? 0 : (v > kTopkListCap ? kTopkListCap : v));
}

// Largest number of probing tokens for which a chunk of a wave of nq queries takes the narrow
// scan: kNarrowMax for waves of at most kNarrowWave queries, where most probed chunks have few
// probing tokens and the wide scan's 16-token tiles would be mostly padding; 0 (every chunk
// wide) for larger waves, where the narrow scan measured slower on the same chunks.
// WARP_NARROW_MAX sets it for every wave (0 sends every chunk to the wide scan); results do
// not depend on it.
int32_t narrow_max(int32_t nq) {
    int64_t v = nq <= kNarrowWave ? kNarrowMax : 0;
    if (const char* s = std::getenv("WARP_NARROW_MAX")) v = std::atoll(s);
    return (int32_t)(v < 0 ? 0 : (v > 4096 ? 4096 : v));
}

hipEvent_t take_event(warp_index* idx) {
    if (!idx->ev_pool.empty()) {
        hipEvent_t e = idx->ev_pool.back();
        idx->ev_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    (void)hipEventCreate(&e);
    return e;
}

void settle_timings(warp_index* idx) {
    const size_t g = kStages + 1;
    for (size_t i = 0; i + g <= idx->ev_pending.size(); i += g) {
        for (int s = 0; s < kStages; ++s) {
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, idx->ev_pending[i + s], idx->ev_pending[i + s + 1]) == hipSuccess) {
                idx->stage_ms[s] += ms;
                idx->stage_launches[s] += 1;
            }
        }
    }
    for (hipEvent_t e : idx->ev_pending) idx->ev_pool.push_back(e);
    idx->ev_pending.clear();
}

struct SearchOut {
    int32_t* ids;
    float* scores;
    int64_t* fixed;
    int32_t* counts;
    int32_t* sel;
    int64_t* m;
    uint32_t* bitmap;
    int64_t* scored;
};

// Scratch of one wave: the device memory its kernels use besides the index and the outputs.
struct WaveScratch {
    uint16_t* filter;
    int32_t *sel, *base;
    int64_t *seg_pref, *m_fixed;
    uint32_t *tokmax, *tokcnt;
    const uint32_t* q_epoch;  // null: cells hold t + 2^31 and the fold resets what it reads
    int32_t* doc_len;
    uint64_t *keys, *qpart;
    int32_t *ccount, *cursor, *pair_start, *plist;
    int64_t* coff;
    int8_t* qdig;
    int4 *list_rec, *list_rec2;
    int64_t *list_item, *cblk;
    uint32_t* scan_queue;
    void *full_sel, *full_topk;  // sort scratch of the sorting selection and of k > kMaxK
    unsigned long long* sel_hist;  // split selection: histograms, band lists and counts of up
    int32_t *sel_lists, *sel_cnt;  // to split_cap tokens
    int64_t split_cap;
};

// The index's own scratch (grown by reserve()).
WaveScratch index_scratch(warp_index* idx) {
    WaveScratch w{};
    w.filter = (uint16_t*)idx->filter.p;
    w.sel = (int32_t*)idx->sel.p;
    w.base = (int32_t*)idx->base.p;
    w.seg_pref = (int64_t*)idx->seg_pref.p;
    w.m_fixed = (int64_t*)idx->m_fixed.p;
    w.tokmax = (uint32_t*)idx->tokmax.p;
    const bool epochs = idx->scoring == WARP_SCORING_PAPER && idx->tab_epochs != 0;
    w.q_epoch = epochs ? (const uint32_t*)idx->q_epoch.p : nullptr;
    w.tokcnt = idx->scoring == WARP_SCORING_EQ1_LITERAL ? (uint32_t*)idx->tokcnt.p : nullptr;
    w.doc_len = (int32_t*)idx->doc_len.p;
    w.keys = (uint64_t*)idx->keys.p;
    w.qpart = (uint64_t*)idx->qpart.p;
    w.ccount = (int32_t*)idx->ccount.p;
    w.cursor = (int32_t*)idx->cursor.p;
    w.pair_start = (int32_t*)idx->pair_start.p;
    w.coff = (int64_t*)idx->coff.p;
    w.plist = (int32_t*)idx->plist.p;
    w.qdig = (int8_t*)idx->qdig.p;
    w.list_rec = (int4*)idx->list_rec.p;
    w.list_item = (int64_t*)idx->list_item.p;
    w.list_rec2 = (int4*)idx->list_rec2.p;
    w.cblk = (int64_t*)idx->cblk.p;
    w.scan_queue = (uint32_t*)idx->scan_queue.p;
    w.full_sel = idx->full_sel.p;
    w.full_topk = idx->full_topk.p;
    w.sel_hist = (unsigned long long*)idx->sel_hist.p;
    w.sel_lists = (int32_t*)idx->sel_lists.p;
    w.sel_cnt = (int32_t*)idx->sel_cnt.p;
    // tokens that all three buffers hold (an unused buffer keeps a 16-byte stub)
    w.split_cap = (int64_t)std::min({idx->sel_hist.bytes / ((size_t)kSelBins * 8),
                                     idx->sel_lists.bytes / ((size_t)2 * kSelCap * 4), idx->sel_cnt.bytes / 8});
    return w;
}

// Enqueue the kernels of one wave (queries [q0, q0 + nq) of the search) on `s`. With epochs,
// the host's copy of the query slots' epochs advances (after zeroing the slots that ran out).
// Returns the first launch error.
hipError_t launch_wave(warp_index* idx, const WaveScratch& w, const float* dq, int32_t q0, int32_t nq, int32_t T,
                 int32_t P, int64_t t_prime, int32_t k, const SearchOut& o, hipStream_t s, bool timed) {
    const int64_t words = ((int64_t)idx->n_docs + 31) / 32;
    WaveArgs a{};
    a.centroids = idx->centroids;
    a.offsets = idx->offsets;
    a.sizes = idx->sizes;
    a.doc_ids = idx->doc_ids;
    a.codes = idx->codes;
    a.weights = idx->weights;
    a.n_c = idx->n_c;
    a.n_docs = idx->n_docs;
    a.nbits = idx->nbits;
    a.queries = dq + (int64_t)q0 * T * kDim;
    a.n_q = nq;
    a.n_qtok = T;
    a.nprobe = P;
    a.k = k;
    a.t_prime = t_prime;
    a.filter_bins = w.filter;
    a.sel = w.sel;
    a.base = w.base;
    a.seg_pref = w.seg_pref;
    a.m_fixed = w.m_fixed;
    a.tokmax = w.tokmax;
    a.q_epoch = w.q_epoch;
    a.tok_w = idx->tab_w;
    a.tokcnt = w.tokcnt;
    a.doc_len = w.doc_len;
    a.keys = w.keys;
    a.qpart = w.qpart;
    a.err = idx->err;
    a.out_ids = o.ids + (int64_t)q0 * k;
    a.out_scores = o.scores + (int64_t)q0 * k;
    a.out_fixed = o.fixed ? o.fixed + (int64_t)q0 * k : nullptr;
    a.out_counts = o.counts ? o.counts + q0 : nullptr;
    a.dbg_sel = o.sel ? o.sel + (int64_t)q0 * T * P : nullptr;
    a.dbg_m = o.m ? o.m + (int64_t)q0 * T : nullptr;
    a.dbg_bitmap = o.bitmap ? o.bitmap + (int64_t)q0 * words : nullptr;
    a.dbg_scored = o.scored ? o.scored + q0 : nullptr;
    a.ccount = w.ccount;
    a.cursor = w.cursor;
    a.pair_start = w.pair_start;
    a.coff = w.coff;
    a.plist = w.plist;
    a.chunk_c = idx->chunk_c;
    a.chunk_k = idx->chunk_k;
    a.n_chunks = idx->n_chunks;
    a.list_rec = w.list_rec;
    a.list_item = w.list_item;
    a.list_n = w.list_item + idx->n_chunks + 1;
    a.list_rec2 = w.list_rec2;
    a.list_n2 = w.list_item + idx->n_chunks + 2;
    a.cblk = w.cblk;
    a.scan_queue = w.scan_queue;
    a.qdig = w.qdig;
    a.scan_grid = idx->scan_grid;
    a.topk_list_cap = topk_list_cap();
    a.narrow_max = narrow_max(nq);
    const int64_t n_tok = (int64_t)nq * T;
    a.sel_slices = n_tok <= w.split_cap ? select_slices(idx, n_tok) : 1;
    a.sel_hist = w.sel_hist;
    a.sel_lists = w.sel_lists;
    a.sel_cnt = w.sel_cnt;

    const bool epochs = w.q_epoch != nullptr;
    hipEvent_t ev[kStages + 1] = {};
    if (timed)
        for (int e = 0; e <= kStages; ++e) ev[e] = take_event(idx);
    auto mark = [&](int e) {
        if (timed) (void)hipEventRecord(ev[e], s);
    };
    mark(0);
    launch_filter_gemm(a.queries, nq * T, idx->centroids, idx->n_c, a.filter_bins, nullptr, s);
    mark(1);
    if (epochs) {  // the slots' next epochs (the preparation applies the same rule on the device),
                   // after zeroing those past the last one
        zero_slots(idx, nq, true, s);
        for (int32_t q = 0; q < nq; ++q)
            idx->slot_ep[q] = idx->slot_ep[q] >= (uint32_t)idx->tab_epochs ? 1u : idx->slot_ep[q] + 1u;
    }
    // the preparation zeroes the cluster token counters that the selection counts into
    launch_wave_prep(a, epochs ? (uint32_t*)idx->q_epoch.p : nullptr, (uint32_t)idx->tab_epochs, s);
    hipError_t err = hipSuccess;
    if (full_select(idx, P)) err = launch_select_full(a, w.full_sel, s);
    else launch_select(a, s);
    mark(2);
    launch_scored(a, s);
    launch_pairing(a, s);
    mark(3);
    launch_scan_mx(a, s);
    launch_scan_narrow(a, idx->narrow_grid, s);
    mark(4);
    launch_fold(a, s);
    mark(5);
    if (k > kMaxK) {
        const hipError_t e = launch_topk_full(a, w.full_topk, s);
        if (err == hipSuccess) err = e;
    } else {
        launch_topk(a, s);
    }
    mark(6);
    if (timed)
        for (int e = 0; e <= kStages; ++e) idx->ev_pending.push_back(ev[e]);
    const hipError_t le = hipGetLastError();
    return err != hipSuccess ? err : le;
}

// Enqueue a whole search on `s`; every pointer is device memory.
int enqueue_search(warp_index* idx, const float* dq, int32_t n_queries, int32_t T, int32_t P,
                   int64_t t_prime, int32_t k, const SearchOut& o, hipStream_t s) {
    if (full_select(idx, P) && (int64_t)T * idx->n_c > ((int64_t)1 << 31))
        return fail(WARP_ENOTSUP, "the sorted selection needs n_qtok * n_centroids <= 2^31");
    const int32_t qw = wave_queries(idx, n_queries, T, P);
    int rc = reserve(idx, qw, T, P, k, s);
    if (rc) return rc;
    const WaveScratch w = index_scratch(idx);
    for (int32_t q0 = 0; q0 < n_queries; q0 += qw) {
        const int32_t nq = n_queries - q0 < qw ? n_queries - q0 : qw;
        const hipError_t le = launch_wave(idx, w, dq, q0, nq, T, P, t_prime, k, o, s, idx->timing);
        if (le != hipSuccess) return fail(WARP_EDEVICE, "kernel launch failed: %s", hipGetErrorString(le));
    }
    return WARP_OK;
}

// The device's error bits since the last check (cleared here), as a status; *bits gets them.
int read_device_errors(warp_index* idx, hipStream_t s, int32_t* bits = nullptr) {
    int32_t err = 0;
    HIP_TRY(hipMemcpyAsync(&err, idx->err, sizeof err, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (idx->timing) settle_timings(idx);
    if (bits) *bits = err;
    if (err) launch_fill_i32(idx->err, 1, 0, s);
    if (err & kErrQueryNorm) idx->tab_force_zero = true;
    if (err & kErrQueryNorm)
        return fail(WARP_EINVAL, "a query token is not finite or has norm > 1 + 1e-3");
    if (err & kErrSelOverflow)
        return fail(WARP_ENOTSUP,
                    "centroid selection overflow: more than %d centroids fall in one selection band "
                    "(degenerate centroid scores)", kSelCap);
    if (err & kErrSelNoCrossing) return fail(WARP_EDEVICE, "centroid selection found no t' crossing");
    return WARP_OK;
}

int search_host(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok, int32_t nprobe,
                int64_t t_prime, int32_t k, int32_t* ids, float* scores, int32_t* counts, int64_t* fixed,
                int32_t* sel, int64_t* m, uint32_t* bitmap, int64_t* scored) {
    int rc = validate_search(idx, queries, n_queries, n_qtok, nprobe, t_prime, k, ids, scores);
    if (rc) return rc;
    std::lock_guard<std::mutex> g(idx->lock);
    HIP_TRY(hipSetDevice(idx->device));
    const int64_t n_tok = (int64_t)n_queries * n_qtok;
    rc = validate_queries_host(queries, n_tok);
    if (rc) return rc;
    const int64_t words = ((int64_t)idx->n_docs + 31) / 32;
    const size_t nk = (size_t)n_queries * k;
    if (!rc) rc = grow_scratch(idx, idx->st_q, (size_t)n_tok * kDim * 4);
    if (!rc) rc = grow_scratch(idx, idx->st_ids, nk * 4);
    if (!rc) rc = grow_scratch(idx, idx->st_scores, nk * 4);
    if (!rc) rc = grow_scratch(idx, idx->st_fixed, nk * 8);
    if (!rc) rc = grow_scratch(idx, idx->st_counts, (size_t)n_queries * 4);
    if (!rc && sel) rc = grow_scratch(idx, idx->st_sel, (size_t)n_tok * nprobe * 4);
    if (!rc && m) rc = grow_scratch(idx, idx->st_m, (size_t)n_tok * 8);
    if (!rc && bitmap) rc = grow_scratch(idx, idx->st_bitmap, (size_t)n_queries * words * 4);
    if (!rc && scored) rc = grow_scratch(idx, idx->st_scored, (size_t)n_queries * 8);
    if (rc) return rc;
    hipStream_t s = idx->stream;
    HIP_TRY(hipMemcpyAsync(idx->st_q.p, queries, (size_t)n_tok * kDim * 4, hipMemcpyHostToDevice, s));
    SearchOut o{(int32_t*)idx->st_ids.p, (float*)idx->st_scores.p, (int64_t*)idx->st_fixed.p,
                (int32_t*)idx->st_counts.p,  sel ? (int32_t*)idx->st_sel.p : nullptr,
                m ? (int64_t*)idx->st_m.p : nullptr, bitmap ? (uint32_t*)idx->st_bitmap.p : nullptr,
                scored ? (int64_t*)idx->st_scored.p : nullptr};
    // A band of the selection that overflowed (a degenerate centroid set) is retried once with the
    // selection that sorts every score, which has no band to overflow.
    int32_t bits = 0;
    for (int attempt = 0; attempt < 2; ++attempt) {
        idx->force_full_select = attempt == 1;
        rc = enqueue_search(idx, (const float*)idx->st_q.p, n_queries, n_qtok, nprobe, t_prime, k, o, s);
        if (!rc) rc = read_device_errors(idx, s, &bits);
        idx->force_full_select = false;
        if (!(rc == WARP_ENOTSUP && (bits & kErrSelOverflow) && attempt == 0)) break;
    }
    if (rc) return rc;
    HIP_TRY(hipMemcpyAsync(ids, o.ids, nk * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(scores, o.scores, nk * 4, hipMemcpyDeviceToHost, s));
    if (fixed) HIP_TRY(hipMemcpyAsync(fixed, o.fixed, nk * 8, hipMemcpyDeviceToHost, s));
    if (counts) HIP_TRY(hipMemcpyAsync(counts, o.counts, (size_t)n_queries * 4, hipMemcpyDeviceToHost, s));
    if (sel) HIP_TRY(hipMemcpyAsync(sel, o.sel, (size_t)n_tok * nprobe * 4, hipMemcpyDeviceToHost, s));
    if (m) HIP_TRY(hipMemcpyAsync(m, o.m, (size_t)n_tok * 8, hipMemcpyDeviceToHost, s));
    if (bitmap)
        HIP_TRY(hipMemcpyAsync(bitmap, o.bitmap, (size_t)n_queries * words * 4, hipMemcpyDeviceToHost, s));
    if (scored) HIP_TRY(hipMemcpyAsync(scored, o.scored, (size_t)n_queries * 8, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return WARP_OK;
}

// The no-allocation scratch laid out for waves of qw queries of T tokens (nprobe P, k results), in
// 256-byte aligned pieces from `base` (null: sizes only); returns the bytes it takes.
size_t noalloc_layout(const warp_index* idx, int32_t qw, int32_t T, int32_t P, int32_t k, bool literal,
                      unsigned char* base, WaveScratch* out) {
    size_t at = 0;
    auto take = [&](size_t bytes) -> void* {
        void* p = base ? (void*)(base + at) : nullptr;
        at += (std::max<size_t>(bytes, 256) + 255) & ~(size_t)255;
        return p;
    };
    const size_t n_tok = (size_t)qw * T, nd = (size_t)idx->n_docs, nc = (size_t)idx->n_c;
    const size_t chunks = (size_t)idx->n_chunks, cblocks = (chunks + kPlanBlock - 1) / kPlanBlock;
    WaveScratch w{};
    w.ccount = (int32_t*)take(nc * 4);
    w.cursor = (int32_t*)take(nc * 4);
    w.pair_start = (int32_t*)take((nc + 1) * 4);
    w.coff = (int64_t*)take((nc + kPairBlock - 1) / kPairBlock * 8);
    w.list_rec = (int4*)take(chunks * 16);
    w.list_rec2 = (int4*)take(chunks * 16);
    w.list_item = (int64_t*)take((chunks + 3) * 8);
    w.cblk = (int64_t*)take(cblocks * 24);
    w.scan_queue = (uint32_t*)take(256);
    w.doc_len = literal ? (int32_t*)take(nd * 4) : nullptr;
    w.filter = (uint16_t*)take(n_tok * nc * 2);
    w.sel = (int32_t*)take(n_tok * P * 4);
    w.base = (int32_t*)take(n_tok * P * 4);
    w.seg_pref = (int64_t*)take(n_tok * (P + 1) * 8);
    w.m_fixed = (int64_t*)take(n_tok * 8);
    w.keys = (uint64_t*)take((size_t)qw * nd * 8);
    w.qpart = (uint64_t*)take((size_t)qw * ((nd + 255) / 256) * 16);
    w.plist = (int32_t*)take(n_tok * P * 8);
    w.qdig = (int8_t*)take(n_tok * kQdigBytes);
    w.tokmax = (uint32_t*)take(n_tok * nd * 4);
    w.tokcnt = literal ? (uint32_t*)take(n_tok * nd * 4) : nullptr;
    w.q_epoch = nullptr;  // cells hold t + 2^31 and the fold resets every cell it reads
    w.full_sel = P > kMaxProbe ? take(select_full_bytes((int64_t)n_tok, idx->n_c)) : nullptr;
    w.full_topk = k > kMaxK ? take(topk_full_bytes(idx->n_docs)) : nullptr;
    w.split_cap = split_tokens(idx, (int64_t)n_tok);
    w.sel_hist = (unsigned long long*)take((size_t)w.split_cap * kSelBins * 8);
    w.sel_lists = (int32_t*)take((size_t)w.split_cap * 2 * kSelCap * 4);
    w.sel_cnt = (int32_t*)take((size_t)w.split_cap * 2 * 4);
    if (out) *out = w;
    return at;
}

}  // namespace

extern "C" {

int warp_search_noalloc(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok, int32_t nprobe,
                        int64_t t_prime, int32_t k, int32_t* out_doc_ids, float* out_scores, int32_t* out_counts,
                        int64_t* out_fixed_scores, void* hip_stream) {
    int rc = validate_search(idx, queries, n_queries, n_qtok, nprobe, t_prime, k, out_doc_ids, out_scores);
    if (rc) return rc;
    std::lock_guard<std::mutex> g(idx->lock);
    HIP_TRY(hipSetDevice(idx->device));
    unsigned char* base = noalloc_scratch(idx->device);
    if (!base) return fail(WARP_EDEVICE, "no-allocation scratch of device %d is not bound", idx->device);
    const bool literal = idx->scoring == WARP_SCORING_EQ1_LITERAL;
    const size_t one = noalloc_layout(idx, 1, n_qtok, nprobe, k, literal, nullptr, nullptr);
    if (one > kNoAllocBytes)
        return fail(WARP_ENOMEM,
                    "warp_search_noalloc: one query of %d tokens on this index needs %zu bytes of scratch; "
                    "the static scratch holds %zu (use warp_search_async)", n_qtok, one, kNoAllocBytes);
    if (nprobe > kMaxProbe && (int64_t)n_qtok * idx->n_c > ((int64_t)1 << 31))
        return fail(WARP_ENOTSUP, "nprobe above %d needs n_qtok * n_centroids <= 2^31", kMaxProbe);
    // the largest wave that fits (the layout grows with the wave); the exact selection
    // sorts at most 2^31 scores per wave
    int32_t lo = 1, hi = n_queries;
    if (nprobe > kMaxProbe) hi = (int32_t)std::min<int64_t>(hi, ((int64_t)1 << 31) / ((int64_t)n_qtok * idx->n_c));
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo + 1) / 2;
        if (noalloc_layout(idx, mid, n_qtok, nprobe, k, literal, nullptr, nullptr) <= kNoAllocBytes) lo = mid;
        else hi = mid - 1;
    }
    const int32_t qw = lo;
    WaveScratch w{};
    noalloc_layout(idx, qw, n_qtok, nprobe, k, literal, base, &w);
    hipStream_t s = (hipStream_t)hip_stream;
    // the array keeps what the last call left: the token-max cells (and counts) start at
    // zero; each wave's fold then resets every cell it reads
    launch_zero_cells(w.tokmax, (int64_t)qw * n_qtok * idx->n_docs, s);
    if (literal) {
        launch_zero_cells(w.tokcnt, (int64_t)qw * n_qtok * idx->n_docs, s);
        launch_doc_len(idx->doc_ids, idx->n_emb, w.doc_len, idx->n_docs, s);
    }
    SearchOut o{out_doc_ids, out_scores, out_fixed_scores, out_counts, nullptr, nullptr, nullptr, nullptr};
    for (int32_t q0 = 0; q0 < n_queries; q0 += qw) {
        const int32_t nq = n_queries - q0 < qw ? n_queries - q0 : qw;
        const hipError_t le = launch_wave(idx, w, queries, q0, nq, n_qtok, nprobe, t_prime, k, o, s, false);
        if (le != hipSuccess) return fail(WARP_EDEVICE, "kernel launch failed: %s", hipGetErrorString(le));
    }
    return WARP_OK;
}

int warp_fixed_point_bits(void) { return kFrac; }

const char* warp_last_error(void) { return g_err.c_str(); }

int warp_t_prime_policy(int64_t n_embeddings, double c, int64_t t_max, int64_t* out) {
    if (!out) return fail(WARP_EINVAL, "out is null");
    if (n_embeddings < 0) return fail(WARP_EINVAL, "n_embeddings must be >= 0");
    if (!(c >= 0.0) || !std::isfinite(c)) return fail(WARP_EINVAL, "c must be finite and >= 0");
    if (t_max < 0) return fail(WARP_EINVAL, "t_max must be >= 0");
    const double t = std::floor(c * std::sqrt((double)n_embeddings));
    *out = t >= (double)t_max ? t_max : (int64_t)t;
    return WARP_OK;
}

int warp_kmeans_sample_size(int64_t n_passages, double c, int64_t* out) {
    if (!out) return fail(WARP_EINVAL, "out is null");
    if (n_passages < 0) return fail(WARP_EINVAL, "n_passages must be >= 0");
    if (!(c >= 0.0) || !std::isfinite(c)) return fail(WARP_EINVAL, "c must be finite and >= 0");
    const double k = std::ceil(c * std::sqrt((double)n_passages));
    *out = k >= (double)n_passages ? n_passages : (int64_t)k;
    return WARP_OK;
}

int warp_index_load(const float* centroids, int32_t n_centroids, int32_t dim, const int64_t* cluster_offsets,
                    const int32_t* doc_ids, const uint8_t* codes, int32_t nbits, const float* bucket_weights,
                    int32_t n_docs, warp_index** out) {
    return load_common(centroids, n_centroids, dim, cluster_offsets, doc_ids, codes, nbits, bucket_weights,
                       n_docs, out, false);
}

int warp_index_load_device(const float* centroids, int32_t n_centroids, int32_t dim,
                           const int64_t* cluster_offsets, const int32_t* doc_ids, const uint8_t* codes,
                           int32_t nbits, const float* bucket_weights, int32_t n_docs, warp_index** out) {
    return load_common(centroids, n_centroids, dim, cluster_offsets, doc_ids, codes, nbits, bucket_weights,
                       n_docs, out, true);
}

void warp_index_free(warp_index* idx) {
    if (!idx) return;
    {
        std::lock_guard<std::mutex> g(g_live_lock);
        if (live_handles().erase(idx) == 0) {  // never loaded, or already freed: nothing to do
            g_err = "warp_index_free: invalid or already freed index handle";
            return;
        }
    }
    destroy_index(idx);
}

int warp_index_info(const warp_index* idx, int32_t* n_centroids, int64_t* n_embeddings, int32_t* n_docs,
                    int32_t* nbits) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    if (n_centroids) *n_centroids = idx->n_c;
    if (n_embeddings) *n_embeddings = idx->n_emb;
    if (n_docs) *n_docs = idx->n_docs;
    if (nbits) *nbits = idx->nbits;
    return WARP_OK;
}

int warp_search(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok, int32_t nprobe,
                int64_t t_prime, int32_t k, int32_t* out_doc_ids, float* out_scores, int32_t* out_counts) {
    return search_host(idx, queries, n_queries, n_qtok, nprobe, t_prime, k, out_doc_ids, out_scores, out_counts,
                       nullptr, nullptr, nullptr, nullptr, nullptr);
}

int warp_search_debug(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok, int32_t nprobe,
                      int64_t t_prime, int32_t k, int32_t* out_doc_ids, float* out_scores, int32_t* out_counts,
                      int64_t* out_fixed_scores, int32_t* sel, int64_t* m_fixed, uint32_t* cand_bitmap,
                      int64_t* n_scored) {
    return search_host(idx, queries, n_queries, n_qtok, nprobe, t_prime, k, out_doc_ids, out_scores, out_counts,
                       out_fixed_scores, sel, m_fixed, cand_bitmap, n_scored);
}

int warp_search_async(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok, int32_t nprobe,
                      int64_t t_prime, int32_t k, int32_t* out_doc_ids, float* out_scores, int32_t* out_counts,
                      int64_t* out_fixed_scores, void* hip_stream) {
    int rc = validate_search(idx, queries, n_queries, n_qtok, nprobe, t_prime, k, out_doc_ids, out_scores);
    if (rc) return rc;
    std::lock_guard<std::mutex> g(idx->lock);
    HIP_TRY(hipSetDevice(idx->device));
    hipStream_t s = (hipStream_t)hip_stream;
    SearchOut o{out_doc_ids, out_scores, out_fixed_scores, out_counts, nullptr, nullptr, nullptr, nullptr};
    return enqueue_search(idx, queries, n_queries, n_qtok, nprobe, t_prime, k, o, s);
}

int warp_index_sync(warp_index* idx, void* hip_stream) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    std::lock_guard<std::mutex> g(idx->lock);
    HIP_TRY(hipSetDevice(idx->device));
    return read_device_errors(idx, (hipStream_t)hip_stream);
}

int warp_centroid_filter_scores(warp_index* idx, const float* queries, int32_t n_tok, float* out) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    if (!queries || !out || n_tok < 1) return fail(WARP_EINVAL, "bad arguments");
    std::lock_guard<std::mutex> g(idx->lock);
    HIP_TRY(hipSetDevice(idx->device));
    DevBuf q, f;
    int rc = grow(q, (size_t)n_tok * kDim * 4);
    if (!rc) rc = grow(f, (size_t)n_tok * idx->n_c * 4);
    if (!rc) {
        hipStream_t s = idx->stream;
        if (hipMemcpyAsync(q.p, queries, (size_t)n_tok * kDim * 4, hipMemcpyHostToDevice, s) != hipSuccess)
            rc = fail(WARP_EDEVICE, "copy failed");
        if (!rc) launch_filter_gemm((const float*)q.p, n_tok, idx->centroids, idx->n_c, nullptr, (float*)f.p, s);
        if (!rc && (hipMemcpyAsync(out, f.p, (size_t)n_tok * idx->n_c * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
                    hipStreamSynchronize(s) != hipSuccess))
            rc = fail(WARP_EDEVICE, "filter scores failed");
    }
    release(q);
    release(f);
    return rc;
}

int warp_build_index(const float* tokens, const int32_t* token_docs, int64_t n_tokens, int32_t n_docs,
                     const float* init_centroids, int32_t n_centroids, const int64_t* sample_ids, int64_t n_sample,
                     int32_t iterations, int32_t nbits, int64_t n_quant, float* centroids, int64_t* cluster_offsets,
                     int32_t* doc_ids, uint8_t* codes, float* bucket_weights, float* bucket_cutoffs,
                     int32_t* assignment) {
    if (!tokens || !token_docs || !init_centroids || !sample_ids || !centroids || !cluster_offsets || !doc_ids ||
        !codes || !bucket_weights || !bucket_cutoffs)
        return fail(WARP_EINVAL, "null pointer argument");
    if (n_tokens < 1 || n_tokens > INT32_MAX / 2) return fail(WARP_EINVAL, "n_tokens must be in [1, 2^30]");
    if (n_docs < 1 || n_docs > kMaxDocs) return fail(WARP_EINVAL, "n_docs must be in [1, 2^24]");
    if (n_centroids < 1 || n_centroids > (1 << 24)) return fail(WARP_EINVAL, "n_centroids must be in [1, 2^24]");
    if (nbits != 1 && nbits != 2 && nbits != 4 && nbits != 8)
        return fail(WARP_EINVAL, "nbits must be 1, 2, 4 or 8 (got %d)", nbits);
    if (iterations < 0 || iterations > 10000) return fail(WARP_EINVAL, "iterations must be in [0, 10000]");
    if (n_sample < 1 || n_sample > (1 << 23)) return fail(WARP_EINVAL, "n_sample must be in [1, 2^23]");
    if (n_quant < 1 || n_quant > n_tokens || n_quant > INT32_MAX / kDim)
        return fail(WARP_EINVAL, "n_quant must be in [1, min(n_tokens, 2^24)]");
    int rc = check_device();
    if (rc) return rc;
    const int64_t n_c = n_centroids;
    // host checks of the small inputs
    std::vector<float> hC((size_t)n_c * kDim);
    std::vector<int64_t> hS((size_t)n_sample);
    HIP_TRY(hipMemcpy(hC.data(), init_centroids, hC.size() * 4, hipMemcpyDefault));
    HIP_TRY(hipMemcpy(hS.data(), sample_ids, hS.size() * 8, hipMemcpyDefault));
    for (int64_t c = 0; c < n_c; ++c) {
        double ss = 0;
        for (int d = 0; d < kDim; ++d) {
            const float v = hC[(size_t)c * kDim + d];
            if (!std::isfinite(v)) return fail(WARP_EINVAL, "starting vector %lld is not finite", (long long)c);
            ss += (double)v * v;
        }
        if (!(ss > 0.0) || !std::isfinite(ss))
            return fail(WARP_EINVAL, "starting vector %lld is zero or too large", (long long)c);
    }
    for (int64_t i = 0; i < n_sample; ++i)
        if (hS[i] < 0 || hS[i] >= n_tokens) return fail(WARP_EINVAL, "sample id %lld is out of range", (long long)i);

    hipStream_t s = nullptr;
    HIP_TRY(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));
    struct Scratch {
        DevBuf err, assign, scores, xs, assign_s, sums, counts, resid, sorted, temp, perm_in, perm, keys;
        ~Scratch() {
            for (DevBuf* b : {&err, &assign, &scores, &xs, &assign_s, &sums, &counts, &resid, &sorted, &temp,
                              &perm_in, &perm, &keys})
                release(*b);
        }
    } w;
    auto done = [&](int code) {
        (void)hipStreamSynchronize(s);
        (void)hipStreamDestroy(s);
        return code;
    };
    const int64_t N = n_tokens;
    const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(N, ((int64_t)1 << 31) / (n_c * 4)));
    size_t tb = 0, t1 = 0, t2 = 0, t3 = 0;
    if (!rc) rc = grow(w.err, 4);
    if (!rc && !assignment) rc = grow(w.assign, (size_t)N * 4);
    if (!rc) rc = grow(w.scores, (size_t)chunk * n_c * 4);
    if (!rc) rc = grow(w.xs, (size_t)n_sample * kDim * 4);
    if (!rc) rc = grow(w.assign_s, (size_t)n_sample * 4);
    if (!rc) rc = grow(w.sums, (size_t)n_c * kDim * 8);
    if (!rc) rc = grow(w.counts, ((size_t)n_c + 1) * 8);
    if (!rc) rc = grow(w.resid, (size_t)n_quant * kDim * 4);
    if (!rc) rc = grow(w.sorted, (size_t)n_quant * kDim * 4);
    if (!rc) rc = grow(w.perm_in, (size_t)N * 8);
    if (!rc) rc = grow(w.perm, (size_t)N * 8);
    if (!rc) rc = grow(w.keys, (size_t)N * 4);
    if (rc) return done(rc);
    int end_bit = 1;
    while (end_bit < 31 && ((int64_t)1 << end_bit) < n_c) ++end_bit;
    if (sort_floats(nullptr, &t1, nullptr, nullptr, n_quant * kDim, s) != hipSuccess ||
        sort_by_cluster(nullptr, &t2, nullptr, nullptr, nullptr, nullptr, N, end_bit, s) != hipSuccess ||
        exclusive_sum_u64(nullptr, &t3, nullptr, nullptr, n_c + 1, s) != hipSuccess)
        return done(fail(WARP_EDEVICE, "device primitive sizing failed"));
    tb = std::max(t1, std::max(t2, t3));
    rc = grow(w.temp, tb);
    if (rc) return done(rc);
    int32_t* err = (int32_t*)w.err.p;
    int32_t* assign = assignment ? assignment : (int32_t*)w.assign.p;

    // inputs: finite tokens of norm <= 1 + 1e-3, document ids in range
    launch_fill_i32(err, 1, 0, s);
    launch_check_queries(tokens, N, err, s);
    launch_check_docs(token_docs, N, n_docs, err, s);
    int32_t herr = 0;
    HIP_TRY(hipMemcpyAsync(&herr, err, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (herr & kErrQueryNorm) return done(fail(WARP_EINVAL, "a token is not finite or has norm > 1 + 1e-3"));
    if (herr & kErrDocRange) return done(fail(WARP_EINVAL, "a token's document id is outside [0, n_docs)"));

    HIP_TRY(hipMemcpyAsync(centroids, hC.data(), hC.size() * 4, hipMemcpyHostToDevice, s));
    launch_normalize_rows(centroids, n_centroids, s);  // the starting centroids
    auto assign_rows = [&](const float* x, int64_t n, int32_t* out) {
        for (int64_t t0 = 0; t0 < n; t0 += chunk) {
            const int64_t nt = std::min(chunk, n - t0);
            launch_filter_gemm(x + t0 * kDim, (int32_t)nt, centroids, n_centroids, nullptr, (float*)w.scores.p, s);
            launch_rows_argmax((const float*)w.scores.p, nt, n_centroids, x + t0 * kDim, centroids, out + t0, err, s);
        }
    };
    // k-means on the sample
    float* xs = (float*)w.xs.p;
    launch_gather_rows(tokens, sample_ids, n_sample, xs, s);
    auto* sums = (unsigned long long*)w.sums.p;
    auto* counts = (unsigned long long*)w.counts.p;
    for (int it = 0; it < iterations; ++it) {
        assign_rows(xs, n_sample, (int32_t*)w.assign_s.p);
        launch_fill_i32((int32_t*)sums, n_c * kDim * 2, 0, s);
        launch_fill_i32((int32_t*)counts, (n_c + 1) * 2, 0, s);
        launch_kmeans_accum(xs, (const int32_t*)w.assign_s.p, n_sample, sums, counts, s);
        launch_kmeans_normalize(sums, counts, n_centroids, centroids, s);
    }
    // every token to its nearest centroid; quantiles of the first n_quant tokens' residuals
    assign_rows(tokens, N, assign);
    launch_residuals(tokens, assign, n_quant, centroids, (float*)w.resid.p, s);
    if (sort_floats(w.temp.p, &tb, (const float*)w.resid.p, (float*)w.sorted.p, n_quant * kDim, s) != hipSuccess)
        return done(fail(WARP_EDEVICE, "residual sort failed"));
    launch_pick_quantiles((const float*)w.sorted.p, n_quant * kDim, nbits, bucket_cutoffs, bucket_weights, s);
    // embeddings grouped by cluster in input order, offsets, codes
    launch_iota64((int64_t*)w.perm_in.p, N, s);
    tb = w.temp.bytes;
    if (sort_by_cluster(w.temp.p, &tb, assign, (int32_t*)w.keys.p, (const int64_t*)w.perm_in.p, (int64_t*)w.perm.p, N,
                        end_bit, s) != hipSuccess)
        return done(fail(WARP_EDEVICE, "cluster sort failed"));
    launch_fill_i32((int32_t*)counts, (n_c + 1) * 2, 0, s);
    launch_count_clusters(assign, N, counts, s);
    tb = w.temp.bytes;
    if (exclusive_sum_u64(w.temp.p, &tb, counts, cluster_offsets, n_c + 1, s) != hipSuccess)
        return done(fail(WARP_EDEVICE, "offset scan failed"));
    launch_encode(nbits, tokens, token_docs, assign, (const int64_t*)w.perm.p, N, centroids, bucket_cutoffs, codes,
                  doc_ids, s);
    HIP_TRY(hipMemcpyAsync(&herr, err, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    const hipError_t le = hipGetLastError();
    if (le != hipSuccess) return done(fail(WARP_EDEVICE, "index build failed: %s", hipGetErrorString(le)));
    if (herr & kErrArgOverflow)
        return done(fail(WARP_ENOTSUP, "more than 1024 centroids tie within 2.5 * 2^-13 of a token's best score"));
    return done(WARP_OK);
}

int warp_set_scoring(warp_index* idx, int32_t mode) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    if (mode != WARP_SCORING_PAPER && mode != WARP_SCORING_EQ1_LITERAL)
        return fail(WARP_EINVAL, "unknown scoring mode %d", mode);
    std::lock_guard<std::mutex> g(idx->lock);
    idx->scoring = mode;
    return WARP_OK;
}

int warp_set_timing(warp_index* idx, int32_t enable) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    std::lock_guard<std::mutex> g(idx->lock);
    idx->timing = enable != 0;
    for (int s = 0; s < kStages; ++s) {
        idx->stage_ms[s] = 0;
        idx->stage_launches[s] = 0;
    }
    for (hipEvent_t e : idx->ev_pending) idx->ev_pool.push_back(e);
    idx->ev_pending.clear();
    return WARP_OK;
}

int warp_stage_timings(const warp_index* idx, double* total_ms, int64_t* launches, int32_t n) {
    if (!is_index(idx)) return fail(WARP_EINVAL, "invalid or freed index handle");
    for (int s = 0; s < n && s < kStages; ++s) {
        if (total_ms) total_ms[s] = idx->stage_ms[s];
        if (launches) launches[s] = idx->stage_launches[s];
    }
    return WARP_OK;
}

}  // extern "C"
