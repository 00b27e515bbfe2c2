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

#include <cstdint>

#include "internal.h"

namespace erase {

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

// ---------------------------------------------------------------------------
// Backward: table gradients from the gradient at x.  Entry i (an index
// position) belongs to the bag (t, m) whose range holds it; its global row
// is t * rows + indices[i].  Entries are bucketed by global row with integer
// counters, and each row's entries are summed in increasing entry order, so
// the result does not depend on scheduling.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void erase_bags_bwd_clear(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
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
      atomicAdd(&a.count[gid], 1);
    } else if (a.status) {
      a.status[0] = 1;
    }
  }
  a.gid[i] = gid;
}

// exclusive prefix sum of the counts (one workgroup of 1024 threads)
__global__ __launch_bounds__(1024) void erase_bags_bwd_scan(EmbedBwdArgs a) {
  __shared__ int part[1024];
  const int tid = threadIdx.x;
  const int64_t per = (a.trows + 1023) / 1024;
  const int64_t lo = tid * per, hi = lo + per < a.trows ? lo + per : a.trows;
  int s = 0;
  for (int64_t v = lo; v < hi; ++v) s += a.count[v];
  part[tid] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int x = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  int run = part[tid] - s;
  for (int64_t v = lo; v < hi; ++v) {
    a.start[v] = run;
    run += a.count[v];
  }
}

__global__ __launch_bounds__(256) void erase_bags_bwd_scatter(EmbedBwdArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.nnz) return;
  const int32_t gid = a.gid[i];
  if (gid >= 0) a.bucket[a.start[gid] + atomicAdd(&a.fill[gid], 1)] = (int32_t)i;
}

// one wave per table row: the row's entries in increasing order (each step
// the smallest entry above the last, a wave-wide minimum), their bags' dx
// columns summed in fp32; rows no entry selects are zero.  dim / 4 lanes
// (dim <= 256) own 4 columns each.
template <typename T>
__global__ __launch_bounds__(256) void erase_bags_bwd_rows(EmbedBwdArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * 4 + wave;
  if (g >= a.trows) return;
  const int t = (int)(g / a.rows);
  const int s0 = a.start[g], c = a.count[g];
  const int32_t mine = lane < c ? a.bucket[s0 + lane] : INT32_MAX;
  const bool col = 4 * lane < a.dim;
  const int64_t xc = a.n_dense + (int64_t)t * a.dim + 4 * lane;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  int32_t prev = -1;
  for (int k = 0; k < c; ++k) {
    int32_t cand = INT32_MAX;
    if (c <= 64) {
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
    if (col) {
      const int m = a.owner[cand] % a.M;
      const T* src = static_cast<const T*>(a.dx) + (int64_t)m * a.lddx + xc;
      if constexpr (sizeof(T) == 2) {
        const u32x2s_t w = *reinterpret_cast<const u32x2s_t*>(src);
        acc.x += __uint_as_float(w.x << 16);
        acc.y += __uint_as_float(w.x & 0xffff0000u);
        acc.z += __uint_as_float(w.y << 16);
        acc.w += __uint_as_float(w.y & 0xffff0000u);
      } else {
        const f32x4s_t v = *reinterpret_cast<const f32x4s_t*>(src);
        acc.x += v[0];
        acc.y += v[1];
        acc.z += v[2];
        acc.w += v[3];
      }
    }
  }
  if (col) *reinterpret_cast<float4*>(a.grad + g * a.dim + 4 * lane) = acc;
}

hipError_t launch_embed_bags_backward(int bf16, const EmbedBwdArgs& a, hipStream_t s) {
  if (a.dim % 4 || a.dim > 256 || a.trows <= 0) return hipErrorInvalidValue;
  const int64_t nmax = a.trows > a.nnz ? a.trows : a.nnz;
  hipLaunchKernelGGL(erase_bags_bwd_clear, dim3((unsigned)((nmax + 255) / 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(erase_bags_bwd_owner, dim3((unsigned)(((int64_t)a.M * a.T + 255) / 256)), dim3(256), 0, s, a);
  if (a.nnz > 0) {
    const dim3 ge((unsigned)((a.nnz + 255) / 256));
    hipLaunchKernelGGL(erase_bags_bwd_count, ge, dim3(256), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scan, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(erase_bags_bwd_scatter, ge, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(erase_bags_bwd_scan, dim3(1), dim3(1024), 0, s, a);
  }
  const dim3 gr((unsigned)((a.trows + 3) / 4));
  if (bf16)
    hipLaunchKernelGGL(erase_bags_bwd_rows<uint16_t>, gr, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(erase_bags_bwd_rows<float>, gr, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace erase
