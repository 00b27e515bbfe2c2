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

constexpr int kSmallBucket = 64;  // entries a wave orders from its registers
constexpr int kSortCap = 16384;   // largest bucket sorted in LDS (64 KB)

// ---------------------------------------------------------------------------
// Backward: table gradients from the gradient at x.  Entry i (an index
// position) belongs to the bag (t, m) whose range holds it; its global row
// is t * rows + indices[i].  Entries are bucketed by global row with integer
// counters, and each row's entries are summed in increasing entry order, so
// the result does not depend on scheduling.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void erase_bags_bwd_clear(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i == 0) a.nlarge[0] = 0;
  if (i < a.trows) {
    a.count[i] = 0;
    a.fill[i] = 0;
  }
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

// one thread per entry: global row and its count
__global__ __launch_bounds__(256) void erase_bags_bwd_count(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.nnz) return;
  const int32_t o = a.owner[i];
  int32_t gid = -1;
  if (o >= 0) {
    const int32_t r = a.indices[i];
    if (r >= 0 && r < a.rows) {
      gid = (int32_t)((o / a.M) * a.rows + r);
      // a row whose count passes kSmallBucket is listed once for sorting
      if (atomicAdd(&a.count[gid], 1) == kSmallBucket) a.large[atomicAdd(a.nlarge, 1)] = gid;
    } else if (a.status) {
      a.status[0] = 1;
    }
  }
  a.gid[i] = gid;
}

// Exclusive prefix sum of the counts in three passes: each workgroup scans
// a block of kScanBlock counts (local offsets into start, the block total
// into bsum), one workgroup scans the block totals, and the block offsets
// are added.
constexpr int kScanBlock = 4096;  // 256 threads x 16 counts

__device__ __forceinline__ int block_exclusive_scan(int v, int* part) {
  // exclusive scan of one value per thread over 256 threads (Hillis-Steele in LDS)
  const int tid = threadIdx.x;
  part[tid] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int x = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  const int incl = part[tid];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scan_local(EmbedBwdArgs a) {
  __shared__ int part[256];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * 16;
  int v[16], s = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    v[k] = base + k < a.trows ? a.count[base + k] : 0;
    s += v[k];
  }
  int run = block_exclusive_scan(s, part);
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (base + k < a.trows) a.start[base + k] = run;
    run += v[k];
  }
  if (threadIdx.x == 255) a.bsum[blockIdx.x] = run;
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scan_blocks(EmbedBwdArgs a) {
  __shared__ int part[256];
  const int nb = (int)((a.trows + kScanBlock - 1) / kScanBlock);
  int carry = 0;
  for (int b0 = 0; b0 < nb; b0 += 256) {
    const int b = b0 + (int)threadIdx.x;
    const int v = b < nb ? a.bsum[b] : 0;
    const int ex = block_exclusive_scan(v, part);
    if (b < nb) a.bsum[b] = carry + ex;
    // the chunk's total, from the last thread's inclusive value
    if (threadIdx.x == 255) part[0] = ex + v;
    __syncthreads();
    carry += part[0];
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scan_add(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < a.trows) a.start[i] += a.bsum[i / kScanBlock];
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scatter(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.nnz) return;
  const int32_t gid = a.gid[i];
  if (gid >= 0) a.bucket[a.start[gid] + atomicAdd(&a.fill[gid], 1)] = (int32_t)i;
}

// Buckets of more than kSmallBucket entries are sorted by entry index: one
// workgroup of 1024 threads per listed bucket, a bitonic sort in LDS of up
// to kSortCap entries (larger buckets keep the selection order below).
__global__ __launch_bounds__(1024) void erase_bags_bwd_sort(EmbedBwdArgs a) {
  __shared__ int32_t key[kSortCap];
  if ((int)blockIdx.x >= a.nlarge[0]) return;  // uniform per workgroup
  const int32_t g = a.large[blockIdx.x];
  const int c = a.count[g], s0 = a.start[g];
  if (c > kSortCap) return;
  int n2 = 1;
  while (n2 < c) n2 <<= 1;
  for (int i = threadIdx.x; i < n2; i += 1024) key[i] = i < c ? a.bucket[s0 + i] : INT32_MAX;
  __syncthreads();
  for (int k = 2; k <= n2; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n2; i += 1024) {
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
  for (int i = threadIdx.x; i < c; i += 1024) {
    a.bucket[s0 + i] = key[i];
    a.bagm[s0 + i] = a.owner[key[i]] % a.M;  // the entry's bag (row of dx)
  }
}

// waves walk the table rows (grid-stride); per row the entries in increasing order, their
// bags' dx columns summed in fp32; rows no entry selects are zero.  Small
// buckets: each step the smallest entry above the last (a wave-wide
// minimum over the entries held in registers); sorted buckets: in bucket
// order; buckets too large to sort: the selection over the bucket.  dim / 4
// lanes (dim <= 256) own 4 columns each.
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

template <typename T, int G>
__global__ __launch_bounds__(256) void erase_bags_bwd_rows(EmbedBwdArgs a) {
  constexpr int E = 64 / G;  // entries summed side by side by the lane groups of a sorted bucket
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = lane / G, cq = lane % G;  // lane group, column quad
  const bool col = 4 * cq < a.dim;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t g = (int64_t)blockIdx.x * 4 + wave; g < a.trows; g += nw) {
    const int t = (int)(g / a.rows);
    const int s0 = a.start[g], c = a.count[g];
    const int64_t xc = a.n_dense + (int64_t)t * a.dim + 4 * cq;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c > kSmallBucket && c <= kSortCap) {
      // sorted bucket, bag rows alongside: group q sums entries q, q + E,
      // ... in increasing order, then the groups are added by a fixed butterfly
      // eight entries' loads in flight, added in entry order
      int k = q;
      for (; k + 7 * E < c; k += 8 * E) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = col ? dx4<T>(a, a.bagm[s0 + k + u * E], xc) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int u = 0; u < 8; ++u) add4(acc, v[u]);
      }
      for (; k < c; k += E)
        if (col) add4(acc, dx4<T>(a, a.bagm[s0 + k], xc));
#pragma unroll
      for (int o = G; o < 64; o <<= 1) {
        acc.x += __shfl_xor(acc.x, o, 64);
        acc.y += __shfl_xor(acc.y, o, 64);
        acc.z += __shfl_xor(acc.z, o, 64);
        acc.w += __shfl_xor(acc.w, o, 64);
      }
    } else {
      // small buckets (and buckets too large to sort): each step the smallest
      // entry above the last, a wave-wide minimum; entries held in
      // registers when there are at most 64
      const int32_t mine = lane < c ? a.bucket[s0 + lane] : INT32_MAX;
      int32_t prev = -1;
      for (int k = 0; k < c; ++k) {
        int32_t cand = INT32_MAX;
        if (c <= kSmallBucket) {
          if (mine > prev) cand = mine;
        } else {
          for (int j = lane; j < c; j += 64) {
            const int32_t p = a.bucket[s0 + j];
            if (p > prev && p < cand) cand = p;
          }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) cand = min(cand, __shfl_xor(cand, o, 64));
        prev = cand;
        if (col) add4(acc, dx4<T>(a, a.owner[cand] % a.M, xc));
      }
    }
    if (col && q == 0) *reinterpret_cast<float4*>(a.grad + g * a.dim + 4 * cq) = acc;
  }
}

hipError_t launch_embed_bags_backward(int bf16, const EmbedBwdArgs& a, hipStream_t s) {
  if (a.dim % 4 || a.dim > 256 || a.trows <= 0) return hipErrorInvalidValue;
  const int64_t nmax = a.trows > a.nnz ? a.trows : a.nnz;
  hipLaunchKernelGGL(erase_bags_bwd_clear, dim3((unsigned)((nmax + 255) / 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(erase_bags_bwd_owner, dim3((unsigned)(((int64_t)a.M * a.T + 255) / 256)), dim3(256), 0, s, a);
  if (a.nnz > 0) {
    const dim3 ge((unsigned)((a.nnz + 255) / 256));
    hipLaunchKernelGGL(erase_bags_bwd_count, ge, dim3(256), 0, s, a);
    const unsigned nsb = (unsigned)((a.trows + kScanBlock - 1) / kScanBlock);
    hipLaunchKernelGGL(erase_bags_bwd_scan_local, dim3(nsb), dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scan_blocks, dim3(1), dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scan_add, dim3((unsigned)((a.trows + 255) / 256)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scatter, ge, dim3(256), 0, s, a);
    // at most nnz / (kSmallBucket + 1) rows pass the small-bucket count
    hipLaunchKernelGGL(erase_bags_bwd_sort, dim3((unsigned)(a.nnz / (kSmallBucket + 1) + 1)), dim3(1024), 0, s, a);
  }
  // no entries: the counts are zero and no row reads start
  const dim3 gr((unsigned)std::min<int64_t>((a.trows + 3) / 4, 8192));
  int G = 1;  // lanes per entry: dim / 4 rounded up to a power of two
  while (G < a.dim / 4) G *= 2;
#define ERASE_BAG_ROWS(GG)                                                                   \
  case GG:                                                                                   \
    if (bf16)                                                                                \
      hipLaunchKernelGGL((erase_bags_bwd_rows<uint16_t, GG>), gr, dim3(256), 0, s, a);       \
    else                                                                                     \
      hipLaunchKernelGGL((erase_bags_bwd_rows<float, GG>), gr, dim3(256), 0, s, a);          \
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
