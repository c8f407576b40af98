// Device-wide primitives: a stable LSD radix sort of 32- or 64-bit keys (optionally
// carrying 64-bit values) and an exclusive prefix sum. The index construction (Section
// 4.1) sorts residual components and (cluster, token) pairs with them; the search sorts
// whole score lists with them when n_probe or k exceed what its selection and top-k
// kernels hold.
//
// Radix sort. Each pass sorts by one 8-bit digit, stably, in three launches:
//   1. k_radix_hist: every tile of kSortTile keys counts its digits; the counts go to a
//      digit-major table hist[digit][tile];
//   2. the exclusive prefix sum of that table (below) gives, for every (digit, tile), the
//      position of the tile's first key with that digit;
//   3. k_radix_scatter: every tile walks its keys in order, in rounds of 256 (one per
//      thread), and places each key at its (digit, tile) position plus the number of keys
//      with the same digit before it in the tile: inside a wave, lanes with equal digits
//      are found with eight ballots; the waves of a round are ordered through LDS, and a
//      running count per digit carries over to the next round.
// Passes alternate between the caller's buffers and two buffers in the temporary storage,
// so the result lands in the caller's output.
//
// Prefix sum. Tiles of kScanTile elements: the tile totals, then (recursively) their
// exclusive prefix sum, then every tile's elements with its tile's offset.
//
// Temporary storage follows the convention of the callers: with temp == nullptr a call
// only sets *temp_bytes.
#include <algorithm>

#include "engine.h"

namespace warp {

constexpr int kSortThreads = 256;
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortThreads * kSortItems;  // keys per tile
constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;

// ---------------------------------------------------------------------------- prefix sum

template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T* s_w, T& total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    T x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const T t = __shfl_up(x, off, 64);
        if (lane >= off) x += t;
    }
    if (lane == 63) s_w[w] = x;
    __syncthreads();
    T before = 0;
    total = 0;
#pragma unroll
    for (int i = 0; i < kScanThreads / 64; ++i) {
        before += i < w ? s_w[i] : (T)0;
        total += s_w[i];
    }
    __syncthreads();
    return before + x - v;
}

// tile totals of in[0, n)
template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(const T* __restrict__ in, int64_t n, T* __restrict__ sums) {
    __shared__ T s_w[kScanThreads / 64];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    T v = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) v += base + i < n ? in[base + i] : (T)0;
    T total;
    block_exclusive_scan<T>(v, s_w, total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// out = exclusive prefix of in, each tile offset by offs[tile] (offs null: 0)
template <typename T, typename U>
__global__ __launch_bounds__(kScanThreads) void k_scan_tiles(const T* __restrict__ in, int64_t n,
                                                            const T* __restrict__ offs, U* __restrict__ out) {
    __shared__ T s_w[kScanThreads / 64];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    T v[kScanItems];
    T sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        v[i] = base + i < n ? in[base + i] : (T)0;
        sum += v[i];
    }
    T total;
    T run = block_exclusive_scan<T>(sum, s_w, total) + (offs ? offs[blockIdx.x] : (T)0);
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        if (base + i < n) out[base + i] = (U)run;
        run += v[i];
    }
}

static int64_t scan_tiles(int64_t n) { return (n + kScanTile - 1) / kScanTile; }

// temporary bytes of exclusive_scan over n elements (tile sums of every level)
template <typename T>
static size_t scan_temp_bytes(int64_t n) {
    size_t b = 0;
    for (int64_t m = scan_tiles(n); m > 1; m = scan_tiles(m)) b += ((size_t)m * sizeof(T) + 255) & ~(size_t)255;
    return b + 256;
}

// out[i] = sum of in[0, i)
template <typename T, typename U>
static void exclusive_scan(void* temp, const T* in, U* out, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    const int64_t tiles = scan_tiles(n);
    if (tiles == 1) {
        hipLaunchKernelGGL((k_scan_tiles<T, U>), dim3(1), dim3(kScanThreads), 0, s, in, n, (const T*)nullptr, out);
        return;
    }
    T* sums = (T*)temp;
    void* rest = (char*)temp + (((size_t)tiles * sizeof(T) + 255) & ~(size_t)255);
    hipLaunchKernelGGL((k_scan_reduce<T>), dim3((unsigned)tiles), dim3(kScanThreads), 0, s, in, n, sums);
    exclusive_scan<T, T>(rest, sums, sums, tiles, s);  // in place: each tile reads before it writes
    hipLaunchKernelGGL((k_scan_tiles<T, U>), dim3((unsigned)tiles), dim3(kScanThreads), 0, s, in, n,
                       (const T*)sums, out);
}

hipError_t exclusive_sum_u64(void* temp, size_t* temp_bytes, const unsigned long long* in, int64_t* out,
                             int64_t n, hipStream_t s) {
    if (!temp) {
        *temp_bytes = scan_temp_bytes<unsigned long long>(n);
        return hipSuccess;
    }
    exclusive_scan<unsigned long long, int64_t>(temp, in, out, n, s);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------- radix sort

template <typename K>
__global__ __launch_bounds__(kSortThreads) void k_radix_hist(const K* __restrict__ keys, int64_t n, int shift,
                                                             int64_t tiles, uint32_t* __restrict__ hist) {
    __shared__ uint32_t s_h[256];
    s_h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
        const int64_t j = base + (int64_t)i * kSortThreads + threadIdx.x;
        if (j < n) atomicAdd(&s_h[(uint32_t)(keys[j] >> shift) & 255u], 1u);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * tiles + blockIdx.x] = s_h[threadIdx.x];
}

// offs[digit * tiles + tile]: the tile's first output position for that digit
template <typename K, bool VALS>
__global__ __launch_bounds__(kSortThreads) void k_radix_scatter(const K* __restrict__ keys_in,
                                                                K* __restrict__ keys_out,
                                                                const int64_t* __restrict__ vals_in,
                                                                int64_t* __restrict__ vals_out, int64_t n, int shift,
                                                                int64_t tiles, const uint32_t* __restrict__ offs) {
    constexpr int NW = kSortThreads / 64;
    __shared__ uint32_t s_next[256];      // next output position of each digit in this tile
    __shared__ uint32_t s_wc[NW][256];    // keys of each digit in each wave of the round
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    s_next[tid] = offs[(int64_t)tid * tiles + blockIdx.x];
#pragma unroll
    for (int i = 0; i < NW; ++i) s_wc[i][tid] = 0;
    __syncthreads();
    const unsigned long long lower = (1ull << lane) - 1;
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t j = base + (int64_t)r * kSortThreads + tid;
        const bool in = j < n;
        const K key = in ? keys_in[j] : (K)0;
        const uint32_t dig = (uint32_t)(key >> shift) & 255u;
        // lanes of this wave holding a key with the same digit
        unsigned long long same = __ballot(in);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const unsigned long long ones = __ballot((dig >> b) & 1u);
            same &= ((dig >> b) & 1u) ? ones : ~ones;
        }
        const uint32_t rank = (uint32_t)__popcll(same & lower);
        // the lowest such lane publishes the wave's count of that digit
        if (in && rank == 0) s_wc[w][dig] = (uint32_t)__popcll(same);
        __syncthreads();
        if (in) {
            uint32_t pos = s_next[dig] + rank;
#pragma unroll
            for (int i = 0; i < NW; ++i) pos += i < w ? s_wc[i][dig] : 0u;
            keys_out[pos] = key;
            if (VALS) vals_out[pos] = vals_in[j];
        }
        __syncthreads();
        // advance the running positions past this round, and clear the wave counts
        uint32_t add = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            add += s_wc[i][tid];
            s_wc[i][tid] = 0;
        }
        s_next[tid] += add;
        __syncthreads();
    }
}

static int64_t sort_tiles(int64_t n) { return (n + kSortTile - 1) / kSortTile; }

// temporary storage of a radix sort of n keys of kb bytes (with 64-bit values if vals):
// the two alternate buffers, the digit table, and its prefix sum's temporary storage
static size_t sort_temp_bytes(int64_t n, bool vals, size_t kb = 4) {
    const auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const int64_t tiles = sort_tiles(n);
    return al((size_t)n * kb) + (vals ? al((size_t)n * 8) : 0) + 2 * al((size_t)tiles * 256 * 4) +
           scan_temp_bytes<uint32_t>(tiles * 256);
}

// Stable sort of keys_in by bits [0, end_bit), values carried along (vals_in may be null).
template <typename K>
static hipError_t radix_sort(void* temp, size_t* temp_bytes, const K* keys_in, K* keys_out,
                             const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s) {
    const bool vals = vals_in != nullptr;
    if (!temp) {
        *temp_bytes = sort_temp_bytes(n, vals, sizeof(K));
        return hipSuccess;
    }
    if (n <= 0) return hipSuccess;
    const auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const int64_t tiles = sort_tiles(n);
    char* p = (char*)temp;
    K* kt = (K*)p;
    p += al((size_t)n * sizeof(K));
    int64_t* vt = vals ? (int64_t*)p : nullptr;
    p += vals ? al((size_t)n * 8) : 0;
    uint32_t* hist = (uint32_t*)p;
    p += al((size_t)tiles * 256 * 4);
    uint32_t* offs = (uint32_t*)p;
    p += al((size_t)tiles * 256 * 4);
    void* scan_temp = p;
    const int passes = std::max(1, (end_bit + 7) / 8);
    // pass i reads src and writes dst; the last pass writes the caller's output
    const K* ks = keys_in;
    const int64_t* vs = vals_in;
    for (int i = 0; i < passes; ++i) {
        const bool to_out = ((passes - 1 - i) % 2) == 0;  // so that the last pass lands in keys_out
        K* kd = to_out ? keys_out : kt;
        int64_t* vd = to_out ? vals_out : vt;
        hipLaunchKernelGGL(k_radix_hist<K>, dim3((unsigned)tiles), dim3(kSortThreads), 0, s, ks, n, 8 * i, tiles, hist);
        exclusive_scan<uint32_t, uint32_t>(scan_temp, hist, offs, tiles * 256, s);
        if (vals)
            hipLaunchKernelGGL((k_radix_scatter<K, true>), dim3((unsigned)tiles), dim3(kSortThreads), 0, s, ks, kd, vs,
                               vd, n, 8 * i, tiles, (const uint32_t*)offs);
        else
            hipLaunchKernelGGL((k_radix_scatter<K, false>), dim3((unsigned)tiles), dim3(kSortThreads), 0, s, ks, kd,
                               (const int64_t*)nullptr, (int64_t*)nullptr, n, 8 * i, tiles, (const uint32_t*)offs);
        ks = kd;
        vs = vd;
    }
    return hipGetLastError();
}

// Temporary bytes of sort_u64 / sort_u32 of n keys, with 64-bit values if vals.
size_t sort_u64_temp_bytes(int64_t n, bool vals) { return sort_temp_bytes(n, vals, 8); }
size_t sort_u32_temp_bytes(int64_t n, bool vals) { return sort_temp_bytes(n, vals, 4); }

hipError_t sort_u64(void* temp, size_t* temp_bytes, const uint64_t* keys_in, uint64_t* keys_out,
                    const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s) {
    return radix_sort<uint64_t>(temp, temp_bytes, keys_in, keys_out, vals_in, vals_out, n, end_bit, s);
}

hipError_t sort_u32(void* temp, size_t* temp_bytes, const uint32_t* keys_in, uint32_t* keys_out,
                    const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s) {
    return radix_sort<uint32_t>(temp, temp_bytes, keys_in, keys_out, vals_in, vals_out, n, end_bit, s);
}

// fp32 <-> order-preserving unsigned keys
__global__ void k_float_keys(const float* __restrict__ in, uint32_t* __restrict__ out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t b = __float_as_uint(in[i]);
    out[i] = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__global__ void k_key_floats(const uint32_t* __restrict__ in, float* __restrict__ out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t k = in[i];
    out[i] = __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Ascending fp32 sort (total order of the bit patterns: -0 before +0; no NaNs reach it).
hipError_t sort_floats(void* temp, size_t* temp_bytes, const float* in, float* out, int64_t n, hipStream_t s) {
    const auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    if (!temp) {
        *temp_bytes = 2 * al((size_t)n * 4) + sort_temp_bytes(n, false);
        return hipSuccess;
    }
    if (n <= 0) return hipSuccess;
    uint32_t* a = (uint32_t*)temp;
    uint32_t* b = (uint32_t*)((char*)temp + al((size_t)n * 4));
    void* rest = (char*)temp + 2 * al((size_t)n * 4);
    const unsigned g = (unsigned)((n + 255) / 256);
    hipLaunchKernelGGL(k_float_keys, dim3(g), dim3(256), 0, s, in, a, n);
    size_t tb = 0;
    hipError_t e = radix_sort<uint32_t>(rest, &tb, a, b, nullptr, nullptr, n, 32, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_key_floats, dim3(g), dim3(256), 0, s, b, out, n);
    return hipGetLastError();
}

// Stable sort of (cluster, token) pairs by cluster, keys in [0, 2^end_bit).
hipError_t sort_by_cluster(void* temp, size_t* temp_bytes, const int32_t* keys_in, int32_t* keys_out,
                           const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s) {
    if (!temp) {
        *temp_bytes = sort_temp_bytes(n, true, 4);
        return hipSuccess;
    }
    return radix_sort<uint32_t>(temp, temp_bytes, reinterpret_cast<const uint32_t*>(keys_in),
                                reinterpret_cast<uint32_t*>(keys_out), vals_in, vals_out, n, end_bit, s);
}

}  // namespace warp
