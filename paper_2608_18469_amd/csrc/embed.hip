// Embedding-bag input stage of the CTR workload, written for gfx950.
//
// x[m] = [ log1p(dense[m][0 .. n_dense)) |  sum over the bag of table 0 |
//          ... | sum over the bag of table T-1 | zeros up to x_ld ]
//
// Each bag is summed in fp32 in the order of its index list.  A wave pools
// 64 / G bags at once: G = dim / 4 (rounded up to a power of two) lanes per
// bag, each lane one 16-byte column chunk, so every row load is one
// contiguous, coalesced read of the row.  Up to 8 rows per bag are in flight
// before they are added.  Out-of-range offsets or indices read nothing: they
// contribute zero and set the status word.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>

#include "erase.h"
#include "internal.h"

namespace erase {

// Scratch of erase_embed_bags_backward_noalloc: one array per GPU, created
// with the code object on that GPU and held until the process ends.  In host
// code `scratch` names a host-side stand-in; kernels get its device address
// from bag_scratch_device_ptr().
static __device__ __align__(256) char scratch[ERASE_BAG_SCRATCH_MAX];

hipError_t bag_scratch_device_ptr(void** ptr, size_t* bytes) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = sizeof(scratch);
  return hipSuccess;
}

typedef float f32x4e_t __attribute__((ext_vector_type(4)));
// output columns start after the dense features, so stores are aligned only
// to the element size (gfx950 serves unaligned vector accesses)
typedef float f32x4s_t __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x2s_t __attribute__((ext_vector_type(2), aligned(2)));

__device__ __forceinline__ uint16_t bag_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

template <typename T, int G>
__global__ __launch_bounds__(256) void erase_embed_bags_k(EmbedArgs a) {
  constexpr int BPW = 64 / G;  // bags per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / G, q = lane % G;  // bag of this lane within the wave, column chunk
  const int64_t nbags = (int64_t)a.M * a.T;
  const int64_t bag = ((int64_t)blockIdx.x * 4 + wave) * BPW + g;
  const bool live = bag < nbags;
  const int m = live ? (int)(bag / a.T) : 0, t = live ? (int)(bag % a.T) : 0;
  const bool col = live && 4 * q < a.dim;

  int64_t beg = 0, end = 0;
  bool bad = false;
  if (live) {
    beg = a.offsets[(int64_t)t * (a.M + 1) + m];
    end = a.offsets[(int64_t)t * (a.M + 1) + m + 1];
    if (!(beg >= 0 && beg <= end && end <= a.nnz)) {
      bad = true;
      beg = end = 0;
    }
  }
  const int n = (int)(end - beg);
  const float* tab = a.tables + (int64_t)t * a.rows * a.dim + 4 * q;
  f32x4e_t acc = {0.f, 0.f, 0.f, 0.f};
  // the longest bag of the wave bounds the loop; shorter bags idle
  int nmax = n;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) nmax = max(nmax, __shfl_xor(nmax, o, 64));
  for (int j0 = 0; j0 < nmax; j0 += 8) {
    f32x4e_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u;
      v[u] = f32x4e_t{0.f, 0.f, 0.f, 0.f};
      if (j < n) {
        const int32_t r = a.indices[beg + j];
        if (r >= 0 && r < a.rows) {
          if (col) v[u] = *reinterpret_cast<const f32x4e_t*>(tab + (int64_t)r * a.dim);
        } else {
          bad = true;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (j0 + u < n) acc += v[u];  // in index order
  }
  if (bad && a.status) a.status[0] = 1;
  if (col) {
    T* dst = static_cast<T*>(a.x) + (int64_t)m * a.ldx + a.n_dense + (int64_t)t * a.dim + 4 * q;
    if constexpr (sizeof(T) == 2) {
      const uint32_t lo = (uint32_t)bag_bf16(acc[0]) | ((uint32_t)bag_bf16(acc[1]) << 16);
      const uint32_t hi = (uint32_t)bag_bf16(acc[2]) | ((uint32_t)bag_bf16(acc[3]) << 16);
      *reinterpret_cast<u32x2s_t*>(dst) = u32x2s_t{lo, hi};
    } else {
      *reinterpret_cast<f32x4s_t*>(dst) = f32x4s_t{acc[0], acc[1], acc[2], acc[3]};
    }
  }
  // the lanes of a row's first table also write its dense features and the
  // zero padding beyond the pooled columns
  if (live && t == 0) {
    T* row = static_cast<T*>(a.x) + (int64_t)m * a.ldx;
    for (int j = q; j < a.n_dense; j += G) {
      const float d = log1pf(a.dense[(int64_t)m * a.n_dense + j]);
      if constexpr (sizeof(T) == 2)
        row[j] = bag_bf16(d);
      else
        row[j] = d;
    }
    const int64_t k0 = a.n_dense + (int64_t)a.T * a.dim;
    for (int64_t k = k0 + q; k < a.ldx; k += G) row[k] = T(0);
  }
}

hipError_t launch_embed_bags(int bf16, const EmbedArgs& a, hipStream_t s) {
  const int c = (a.dim + 3) / 4;
  int G = 1;
  while (G < c) G *= 2;
  const int64_t nbags = (int64_t)a.M * a.T;
  const int64_t per_wg = 4 * (64 / G);
  dim3 grid((unsigned)((nbags + per_wg - 1) / per_wg)), block(256);
#define ERASE_BAGS(GG)                                                                     \
  case GG:                                                                                 \
    if (bf16)                                                                              \
      hipLaunchKernelGGL((erase_embed_bags_k<uint16_t, GG>), grid, block, 0, s, a);        \
    else                                                                                   \
      hipLaunchKernelGGL((erase_embed_bags_k<float, GG>), grid, block, 0, s, a);           \
    break;
  switch (G) {
    ERASE_BAGS(1)
    ERASE_BAGS(2)
    ERASE_BAGS(4)
    ERASE_BAGS(8)
    ERASE_BAGS(16)
    ERASE_BAGS(32)
    ERASE_BAGS(64)
    default: return hipErrorInvalidValue;
  }
#undef ERASE_BAGS
  return hipGetLastError();
}

constexpr int kSmallBucket = 64;  // entries a wave sorts in its registers
constexpr int kSortCap = 16384;   // largest bucket sorted in LDS (64 KB)

// ---------------------------------------------------------------------------
// Backward: table gradients from the gradient at x.  Entry i (an index
// position) belongs to the bag (t, m) whose range holds it; its global row
// is t * rows + indices[i].  Entries are bucketed by global row (counts,
// an exclusive scan, then each entry to its slot), every bucket is put in
// increasing entry order, and each row is summed in a fixed order of its
// entries, so the result does not depend on scheduling:
//  * rows of at most 64 entries: one wave; entries sorted across its lanes,
//    entry k to lane group k mod (64/G) (G lanes of 4 columns cover a row),
//    each group adding its entries in order, the groups then combined by a
//    fixed butterfly;
//  * rows of 65..1024 entries: one workgroup of 256 threads, and rows of
//    1025..16384 entries one of 1024 threads; entries sorted in LDS (a
//    bitmap over their range, or a bitonic sort), entry
//    k to lane group k mod (threads/G), the groups' partial rows then added
//    in group order;
//  * larger rows: increasing entry order, by repeated selection (correct but
//    slow; no workload here has such a row);
//  * rows no entry selects: zero, written by the waves that scan the counts.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void erase_bags_bwd_clear(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i == 0) {
    a.nlarge[0] = 0;  // rows listed for the large-bucket kernels
    a.nlarge[1] = 0;  // rows of 1..kSmallBucket entries (set by the scans)
  }
  if (i < a.trows) a.count[i] = 0;
  if (i < a.nnz) a.owner[i] = -1;
}

// one thread per bag: its entries' owner
__global__ __launch_bounds__(256) void erase_bags_bwd_owner(EmbedBwdArgs a) {
  const int64_t bag = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (bag >= (int64_t)a.M * a.T) return;
  const int t = (int)(bag / a.M), m = (int)(bag % a.M);
  const int64_t beg = a.offsets[(int64_t)t * (a.M + 1) + m], end = a.offsets[(int64_t)t * (a.M + 1) + m + 1];
  if (!(beg >= 0 && beg <= end && end <= a.nnz)) {
    if (a.status) a.status[0] = 1;
    return;
  }
  for (int64_t i = beg; i < end; ++i) a.owner[i] = (int32_t)bag;
}

// Each entry's global row, and its slot in the row's bucket.  A workgroup
// takes kCountTile entries (kCountPer per thread) and first counts their
// rows in an LDS hash table, so each row it holds takes one addition to its
// global counter per workgroup (Zipf-hot rows occur in most workgroups, and
// the additions to one counter are serialised).  Slots need only be distinct
// within a bucket (every bucket is sorted by entry before it is summed): an
// entry's slot is its row's base from that addition plus its rank from the
// LDS count.
constexpr int kCountPer = 8, kCountTile = 256 * kCountPer, kHashSlots = 2 * kCountTile;
__global__ __launch_bounds__(256) void erase_bags_bwd_count(EmbedBwdArgs a) {
  __shared__ int32_t hkey[kHashSlots];  // global row, -1: empty
  __shared__ int32_t hval[kHashSlots];  // the row's entries in this tile, then its base
  const int tid = threadIdx.x;
  for (int h = tid; h < kHashSlots; h += 256) {
    hkey[h] = -1;
    hval[h] = 0;
  }
  __syncthreads();
  const int64_t i0 = (int64_t)blockIdx.x * kCountTile + tid;
  int32_t gid[kCountPer], hs[kCountPer], rk[kCountPer];
#pragma unroll
  for (int u = 0; u < kCountPer; ++u) {
    const int64_t i = i0 + u * 256;
    gid[u] = -1;
    hs[u] = 0;
    rk[u] = 0;
    if (i < a.nnz) {
      const int32_t o = a.owner[i];
      if (o >= 0) {
        const int32_t r = a.indices[i];
        if (r >= 0 && r < a.rows) {
          gid[u] = (int32_t)((o / a.M) * a.rows + r);
        } else if (a.status) {
          a.status[0] = 1;
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kCountPer; ++u) {
    if (gid[u] < 0) continue;
    // open addressing: at most kCountTile keys in 2 kCountTile slots
    int h = (int)(((uint32_t)gid[u] * 0x9E3779B1u) >> 20) & (kHashSlots - 1);
    while (true) {
      const int32_t prev = atomicCAS(&hkey[h], -1, gid[u]);
      if (prev == -1 || prev == gid[u]) break;
      h = (h + 1) & (kHashSlots - 1);
    }
    hs[u] = h;
    rk[u] = atomicAdd(&hval[h], 1);
  }
  __syncthreads();
  for (int h = tid; h < kHashSlots; h += 256) {
    const int32_t g = hkey[h];
    if (g < 0) continue;
    const int k = hval[h];
    const int32_t base = atomicAdd(&a.count[g], k);
    // a row whose count passes kSmallBucket is listed once (exactly one
    // addition crosses the threshold)
    if (base <= kSmallBucket && base + k > kSmallBucket) a.large[atomicAdd(a.nlarge, 1)] = g;
    hval[h] = base;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kCountPer; ++u) {
    const int64_t i = i0 + u * 256;
    if (i < a.nnz) {
      a.gid[i] = gid[u];
      a.slot[i] = gid[u] >= 0 ? hval[hs[u]] + rk[u] : 0;
    }
  }
}

// Exclusive prefix sums over the table rows in three passes, of the counts
// (each bucket's start) and of the flags of rows with 1..kSmallBucket
// entries (each such row's place in the list the row-sum kernel walks):
// each workgroup sums a block of kScanBlock rows (count offsets into start,
// block totals into bsum and bsum2), one workgroup scans the block totals,
// and a last pass adds the block offsets and writes the list.
constexpr int kScanBlock = 4096;  // 256 threads x 16 rows

__device__ __forceinline__ int block_exclusive_scan(int v, int* part) {
  // exclusive scan of one value per thread over 256 threads: inclusive scans
  // within the waves (lane shifts), then the wave totals through LDS
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) part[w] = x;
  __syncthreads();
  int base = 0;
  for (int k = 0; k < w; ++k) base += part[k];
  __syncthreads();
  return base + x - v;
}

__device__ __forceinline__ bool small_row(int c) { return c > 0 && c <= kSmallBucket; }

// a thread's 16 consecutive rows: four 16-byte accesses when all exist
__device__ __forceinline__ void load16(const int32_t* p, int64_t base, int64_t n, int v[16]) {
  if (base + 16 <= n) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int4 x = reinterpret_cast<const int4*>(p + base)[q];
      v[4 * q] = x.x;
      v[4 * q + 1] = x.y;
      v[4 * q + 2] = x.z;
      v[4 * q + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = base + k < n ? p[base + k] : 0;
  }
}
__device__ __forceinline__ void store16(int32_t* p, int64_t base, int64_t n, const int v[16]) {
  if (base + 16 <= n) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      reinterpret_cast<int4*>(p + base)[q] = make_int4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (base + k < n) p[base + k] = v[k];
  }
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scan_local(EmbedBwdArgs a) {
  __shared__ int part[256];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * 16;
  int v[16], st[16], s = 0, f = 0;
  load16(a.count, base, a.trows, v);
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    s += v[k];
    f += small_row(v[k]) ? 1 : 0;
  }
  int run = block_exclusive_scan(s, part);
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    st[k] = run;
    run += v[k];
  }
  store16(a.start, base, a.trows, st);
  const int fx = block_exclusive_scan(f, part);
  if (threadIdx.x == 255) {
    a.bsum[blockIdx.x] = run;
    a.bsum2[blockIdx.x] = fx + f;
  }
}

__device__ __forceinline__ int scan_totals(int* t, int nb, int* part) {
  // exclusive scan of t[0..nb) in place; returns the total
  int carry = 0;
  for (int b0 = 0; b0 < nb; b0 += 256) {
    const int b = b0 + (int)threadIdx.x;
    const int v = b < nb ? t[b] : 0;
    const int ex = block_exclusive_scan(v, part);
    if (b < nb) t[b] = carry + ex;
    // the chunk's total, from the last thread's inclusive value
    if (threadIdx.x == 255) part[0] = ex + v;
    __syncthreads();
    carry += part[0];
    __syncthreads();
  }
  return carry;
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scan_blocks(EmbedBwdArgs a) {
  __shared__ int part[256];
  const int nb = (int)((a.trows + kScanBlock - 1) / kScanBlock);
  (void)scan_totals(a.bsum, nb, part);
  const int nsmall = scan_totals(a.bsum2, nb, part);
  if (threadIdx.x == 0) a.nlarge[1] = nsmall;
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scan_add(EmbedBwdArgs a) {
  __shared__ int part[256];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * 16;
  const int off = a.bsum[blockIdx.x];
  int f = 0, st[16], c[16];
  bool fl[16];
  load16(a.start, base, a.trows, st);
  load16(a.count, base, a.trows, c);
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    st[k] += off;
    fl[k] = base + k < a.trows && small_row(c[k]);
    f += fl[k] ? 1 : 0;
  }
  store16(a.start, base, a.trows, st);
  int pos = a.bsum2[blockIdx.x] + block_exclusive_scan(f, part);
#pragma unroll
  for (int k = 0; k < 16; ++k)
    if (fl[k]) a.small[pos++] = (int32_t)(base + k);
}

// one thread per entry: into its slot of its row's bucket (no atomics)
__global__ __launch_bounds__(256) void erase_bags_bwd_scatter(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.nnz) return;
  const int32_t gid = a.gid[i];
  if (gid >= 0) a.bucket[a.start[gid] + a.slot[i]] = (int32_t)i;
}

// 4 consecutive dx columns of bag row m, as fp32
template <typename T>
__device__ __forceinline__ float4 dx4(const EmbedBwdArgs& a, int m, int64_t xc) {
  const T* src = static_cast<const T*>(a.dx) + (int64_t)m * a.lddx + xc;
  if constexpr (sizeof(T) == 2) {
    const u32x2s_t w = *reinterpret_cast<const u32x2s_t*>(src);
    return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u), __uint_as_float(w.y << 16),
                       __uint_as_float(w.y & 0xffff0000u));
  } else {
    const f32x4s_t v = *reinterpret_cast<const f32x4s_t*>(src);
    return make_float4(v[0], v[1], v[2], v[3]);
  }
}
__device__ __forceinline__ void add4(float4& a, const float4& b) {
  a.x += b.x;
  a.y += b.y;
  a.z += b.z;
  a.w += b.w;
}

// Buckets of more than kSmallBucket entries (the listed rows): one workgroup
// of NT threads per bucket of LO < c <= HI entries sorts it by entry in LDS
// (up to CAP entries: a bitmap over the bucket's entry range when it spans
// at most 32 kBitWords entries, as on the CTR shape, else a bitonic sort),
// turns the entries into their bag rows, and
// sums the row: lane group q (G lanes, 4 columns each) takes entries q,
// q + NG, ... in order, then the NG partial rows are added in group order.
// Buckets beyond CAP are summed in increasing entry order by repeated
// selection.  Instances: 256 threads for 65..1024 entries, 1024 threads
// above (kSortCap, 16384, sorted).
constexpr int kBitWords = 2048;  // bitmap of the bitmap sort: buckets whose entries span <= 64 Ki

// Minimum over the NT threads of a workgroup (every thread gets it).
template <int NT>
__device__ __forceinline__ int32_t block_min_nt(int32_t v, int32_t* sel) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  if ((threadIdx.x & 63) == 0) sel[threadIdx.x >> 6] = v;
  __syncthreads();
  v = sel[0];
  for (int w = 1; w < NT / 64; ++w) v = min(v, sel[w]);
  __syncthreads();
  return v;
}
// Exclusive prefix sum of one value per thread over the NT threads.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan_nt(int v, int32_t* sel) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sel[w] = x;
  __syncthreads();
  int base = 0;
  for (int k = 0; k < w; ++k) base += sel[k];
  __syncthreads();
  return base + x - v;
}
constexpr int kMidBucket = 1024;
template <typename T, int G, int NT, int CAP>
__global__ __launch_bounds__(NT) void erase_bags_bwd_large(EmbedBwdArgs a, int lo, int hi) {
  constexpr int NG = NT / G;  // lane groups of the workgroup
  static_assert(NG * 4 * G <= CAP, "partial rows fit in the key array");
  __shared__ int32_t key[CAP];
  __shared__ int32_t sel[NT / 64];
  __shared__ uint32_t bits[kBitWords];
  if ((int)blockIdx.x >= a.nlarge[0]) return;  // uniform per workgroup
  const int32_t g = a.large[blockIdx.x];
  const int c = a.count[g], s0 = a.start[g];
  if (c <= lo || c > hi) return;  // the other instance's bucket
  const int tid = threadIdx.x;
  const int q = tid / G, cq = tid % G;
  const bool col = 4 * cq < a.dim;
  const int t = g / a.rows;
  const int64_t xc = a.n_dense + (int64_t)t * a.dim + 4 * cq;
  float* out = a.grad + (int64_t)g * a.dim + 4 * cq;
  if (c > CAP) {
    // increasing entry order by repeated selection: a workgroup-wide minimum
    // of the entries above the last one; group 0 adds
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int32_t prev = -1;
    for (int k = 0; k < c; ++k) {
      int32_t cand = INT32_MAX;
      for (int j = tid; j < c; j += NT) {
        const int32_t p = a.bucket[s0 + j];
        if (p > prev && p < cand) cand = p;
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) cand = min(cand, __shfl_xor(cand, o, 64));
      if ((tid & 63) == 0) sel[tid >> 6] = cand;
      __syncthreads();
      cand = sel[0];
      for (int w = 1; w < NT / 64; ++w) cand = min(cand, sel[w]);
      __syncthreads();
      prev = cand;
      if (q == 0 && col) add4(acc, dx4<T>(a, a.owner[cand] % a.M, xc));
    }
    if (q == 0 && col) *reinterpret_cast<float4*>(out) = acc;
    return;
  }
  constexpr int PER = CAP / NT;  // keys per thread
  // the bucket's entry range
  int32_t e_lo = INT32_MAX, e_hi = -1;
  for (int i = tid; i < c; i += NT) {
    const int32_t p = a.bucket[s0 + i];
    e_lo = min(e_lo, p);
    e_hi = max(e_hi, p);
  }
  e_lo = block_min_nt<NT>(e_lo, sel);
  e_hi = -block_min_nt<NT>(-e_hi, sel);
  const int64_t range = (int64_t)e_hi - e_lo + 1;
  if (range <= 32 * (int64_t)kBitWords) {
    // Bitmap sort (the entries of a bucket are distinct): one bit per entry
    // of the range, then every thread lists the set bits of its run of
    // words, in order, at its place from a scan of the runs' bit counts.
    const int nw = (int)((range + 31) / 32);
    for (int w = tid; w < nw; w += NT) bits[w] = 0u;
    __syncthreads();
    for (int i = tid; i < c; i += NT) {
      const int32_t p = a.bucket[s0 + i] - e_lo;
      atomicOr(&bits[p >> 5], 1u << (p & 31));
    }
    __syncthreads();
    const int per = (nw + NT - 1) / NT, w0 = min(nw, tid * per), w1 = min(nw, w0 + per);
    int cnt = 0;
    for (int w = w0; w < w1; ++w) cnt += __popc(bits[w]);
    int pos = block_exclusive_scan_nt<NT>(cnt, sel);
    for (int w = w0; w < w1; ++w) {
      uint32_t b = bits[w];
      while (b) {
        key[pos++] = e_lo + 32 * w + (__ffs(b) - 1);
        b &= b - 1u;
      }
    }
    __syncthreads();
  } else {
    // bitonic sort of the bucket in LDS
    int n2 = 1;
    while (n2 < c) n2 <<= 1;
    {
      int32_t tmp[PER];  // every load in flight before the LDS stores
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int i = tid + u * NT;
        tmp[u] = i < c ? a.bucket[s0 + i] : INT32_MAX;
      }
#pragma unroll
      for (int u = 0; u < PER; ++u)
        if (tid + u * NT < n2) key[tid + u * NT] = tmp[u];
    }
    __syncthreads();
    for (int k = 2; k <= n2; k <<= 1)
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = tid; i < n2; i += NT) {
          const int l = i ^ j;
          if (l > i) {
            const int32_t x = key[i], y = key[l];
            if (((i & k) == 0) == (x > y)) {
              key[i] = y;
              key[l] = x;
            }
          }
        }
        __syncthreads();
      }
  }
  // entries -> their bag rows (rows of dx), in place (each thread its own keys)
  {
    int32_t tmp[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + u * NT;
      tmp[u] = i < c ? a.owner[key[i]] % a.M : 0;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u)
      if (tid + u * NT < c) key[tid + u * NT] = tmp[u];
  }
  __syncthreads();
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (col) {
    int k = q;
    for (; k + 15 * NG < c; k += 16 * NG) {
      float4 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = dx4<T>(a, key[k + u * NG], xc);
#pragma unroll
      for (int u = 0; u < 16; ++u) add4(acc, v[u]);
    }
    for (; k < c; k += NG) add4(acc, dx4<T>(a, key[k], xc));
  }
  __syncthreads();  // key[] is reused for the partial rows
  float* part = reinterpret_cast<float*>(key);  // [NG][4 G] floats
  if (col) *reinterpret_cast<float4*>(part + q * 4 * G + 4 * cq) = acc;
  __syncthreads();
  if (tid < a.dim) {
    float sum = 0.f;
    for (int w = 0; w < NG; ++w) sum += part[w * 4 * G + tid];
    a.grad[(int64_t)g * a.dim + tid] = sum;
  }
}

// Bitonic sort (ascending) of one value per lane across a wave.
__device__ __forceinline__ int32_t wave_sort(int32_t v, int lane) {
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int32_t o = __shfl_xor(v, j, 64);
      const bool lower = (lane & j) == 0, up = (lane & k) == 0;
      v = (lower == up) ? min(v, o) : max(v, o);
    }
  return v;
}

// Rows no entry selects: zeros, one 16-byte chunk per thread.
__global__ __launch_bounds__(256) void erase_bags_bwd_zero(EmbedBwdArgs a) {
  const int cpr = a.dim / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.trows * cpr) return;
  if (a.count[i / cpr] == 0) {
    // streaming stores: the zeros are not read again by this launch sequence
    typedef float f32x4v_t __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(f32x4v_t{0.f, 0.f, 0.f, 0.f}, reinterpret_cast<f32x4v_t*>(a.grad + 4 * i));
  }
}

// Listed rows of 1..kSmallBucket entries, in groups of 64 / G consecutive
// rows per wave (grid-stride), one row per lane group of G lanes.
//  * When every row of the group has at most 4 entries (92% of the rows
//    with entries on the CTR shape, 73% have one), each lane group sums its
//    own row: its entries sorted in registers, their bag rows and dx slices
//    loaded by the group's lanes, added as (0 + v0 + 0 + v1) ... exactly as
//    the wave path below associates at most 4 entries:
//    ((0 + v0) + (0 + v1)) + ((0 + v2) + (0 + v3)).
//  * Otherwise the group's rows go one after another through the wave path:
//    the row's entries sorted across the lanes, their bag rows looked up in
//    parallel, lane group q adding entries q, q + 64/G, ... in order (eight
//    loads in flight), the groups combined by a fixed butterfly.
// Either way a row's sum depends only on its own entries.  (Loading the next
// row's list entry, count and bucket during the current row's sums measured
// slower: 146 against 131 us on the CTR shape, before the per-group path.)
__device__ __forceinline__ void sort2(int32_t& x, int32_t& y) {
  const int32_t lo = min(x, y), hi = max(x, y);
  x = lo;
  y = hi;
}
template <typename T, int G>
__global__ __launch_bounds__(256) void erase_bags_bwd_rows(EmbedBwdArgs a) {
  constexpr int NGW = 64 / G;  // lane groups per wave
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = lane / G, cq = lane % G;  // lane group, column quad
  const bool col = 4 * cq < a.dim;
  const int n = a.nlarge[1];
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int grp = (int)blockIdx.x * 4 + wave; grp * NGW < n; grp += (int)gridDim.x * 4) {
    if constexpr (NGW >= 4) {
      const int idx = grp * NGW + q;
      const bool has = idx < n;
      const int64_t gq = has ? a.small[idx] : 0;
      const int cn = has ? a.count[gq] : 0, sq = has ? a.start[gq] : 0;
      if (__all(cn <= 4)) {  // wave-uniform
        int32_t e[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) e[k] = k < cn ? a.bucket[sq + k] : INT32_MAX;
        sort2(e[0], e[1]);
        sort2(e[2], e[3]);
        sort2(e[0], e[2]);
        sort2(e[1], e[3]);
        sort2(e[1], e[2]);
        const int64_t xc = a.n_dense + (gq / a.rows) * a.dim + 4 * cq;
        float4 v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int m = k < cn ? a.owner[e[k]] % a.M : 0;
          v[k] = (k < cn && col) ? dx4<T>(a, m, xc) : zero;
        }
        float4 s01 = zero, s1 = zero, s23 = zero, s3 = zero;
        add4(s01, v[0]);
        add4(s1, v[1]);
        add4(s01, s1);
        add4(s23, v[2]);
        add4(s3, v[3]);
        add4(s23, s3);
        add4(s01, s23);
        if (has && col) *reinterpret_cast<float4*>(a.grad + gq * a.dim + 4 * cq) = s01;
        continue;
      }
    }
    for (int j = 0; j < NGW; ++j) {
      const int idx = grp * NGW + j;
      if (idx >= n) break;
      const int64_t g = a.small[idx];
      const int c = a.count[g], s0 = a.start[g];
      const int32_t e = wave_sort(lane < c ? a.bucket[s0 + lane] : INT32_MAX, lane);
      const int m = lane < c ? a.owner[e] % a.M : 0;  // bag row of the lane's entry
      const int t = (int)(g / a.rows);
      const int64_t xc = a.n_dense + (int64_t)t * a.dim + 4 * cq;
      float4 acc = zero;
      for (int k0 = 0; k0 < c; k0 += 8 * NGW) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int k = k0 + u * NGW + q;
          const int mk = __shfl(m, k & 63, 64);
          v[u] = (k < c && col) ? dx4<T>(a, mk, xc) : zero;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) add4(acc, v[u]);
      }
#pragma unroll
      for (int o = G; o < 64; o <<= 1) {
        acc.x += __shfl_xor(acc.x, o, 64);
        acc.y += __shfl_xor(acc.y, o, 64);
        acc.z += __shfl_xor(acc.z, o, 64);
        acc.w += __shfl_xor(acc.w, o, 64);
      }
      if (col && q == 0) *reinterpret_cast<float4*>(a.grad + g * a.dim + 4 * cq) = acc;
    }
  }
}

hipError_t launch_embed_bags_backward(int bf16, const EmbedBwdArgs& a, hipStream_t s) {
  if (a.dim % 4 || a.dim > 256 || a.trows <= 0) return hipErrorInvalidValue;
  const int64_t nmax = a.trows > a.nnz ? a.trows : a.nnz;
  hipLaunchKernelGGL(erase_bags_bwd_clear, dim3((unsigned)((nmax + 255) / 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(erase_bags_bwd_owner, dim3((unsigned)(((int64_t)a.M * a.T + 255) / 256)), dim3(256), 0, s, a);
  if (a.nnz > 0) {
    const dim3 ge((unsigned)((a.nnz + 255) / 256));
    hipLaunchKernelGGL(erase_bags_bwd_count, dim3((unsigned)((a.nnz + kCountTile - 1) / kCountTile)), dim3(256), 0,
                       s, a);
    const unsigned nsb = (unsigned)((a.trows + kScanBlock - 1) / kScanBlock);
    hipLaunchKernelGGL(erase_bags_bwd_scan_local, dim3(nsb), dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scan_blocks, dim3(1), dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scan_add, dim3(nsb), dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scatter, ge, dim3(256), 0, s, a);
  }
  // rows no entry selects (every row when there are no entries): zeros
  hipLaunchKernelGGL(erase_bags_bwd_zero, dim3((unsigned)((a.trows * (a.dim / 4) + 255) / 256)), dim3(256), 0, s, a);
  int G = 1;  // lanes per row: dim / 4 rounded up to a power of two
  while (G < a.dim / 4) G *= 2;
  // listed rows of 1..kSmallBucket entries: at most min(rows, entries)
  const int64_t nsmall_max = std::min<int64_t>(a.trows, std::max<int64_t>(a.nnz, 1));
  const dim3 gr((unsigned)std::min<int64_t>((nsmall_max + 3) / 4, 16384));
  // at most nnz / (kSmallBucket + 1) rows pass the small-bucket count
  const dim3 gl((unsigned)(a.nnz / (kSmallBucket + 1) + 1));
#define ERASE_BAG_ROWS(GG)                                                                                \
  case GG:                                                                                                \
    if (bf16) {                                                                                           \
      if (a.nnz > 0) {                                                                                    \
        hipLaunchKernelGGL((erase_bags_bwd_large<uint16_t, GG, 256, kMidBucket>), gl, dim3(256), 0, s, a,  \
                           kSmallBucket, kMidBucket);                                                     \
        hipLaunchKernelGGL((erase_bags_bwd_large<uint16_t, GG, 1024, kSortCap>), gl, dim3(1024), 0, s, a,  \
                           kMidBucket, INT32_MAX);                                                        \
      }                                                                                                   \
      hipLaunchKernelGGL((erase_bags_bwd_rows<uint16_t, GG>), gr, dim3(256), 0, s, a);                    \
    } else {                                                                                              \
      if (a.nnz > 0) {                                                                                    \
        hipLaunchKernelGGL((erase_bags_bwd_large<float, GG, 256, kMidBucket>), gl, dim3(256), 0, s, a,     \
                           kSmallBucket, kMidBucket);                                                     \
        hipLaunchKernelGGL((erase_bags_bwd_large<float, GG, 1024, kSortCap>), gl, dim3(1024), 0, s, a,     \
                           kMidBucket, INT32_MAX);                                                        \
      }                                                                                                   \
      hipLaunchKernelGGL((erase_bags_bwd_rows<float, GG>), gr, dim3(256), 0, s, a);                       \
    }                                                                                                     \
    break;
  switch (G) {
    ERASE_BAG_ROWS(1)
    ERASE_BAG_ROWS(2)
    ERASE_BAG_ROWS(4)
    ERASE_BAG_ROWS(8)
    ERASE_BAG_ROWS(16)
    ERASE_BAG_ROWS(32)
    ERASE_BAG_ROWS(64)
    default: return hipErrorInvalidValue;
  }
#undef ERASE_BAG_ROWS
  return hipGetLastError();
}

}  // namespace erase
