// HIP kernels of the detached-block training step, written for gfx950
// (CDNA4: 64-wide wavefronts, MFMA matrix cores, 160 KB LDS per CU).
//
//  * erase_{fwd,fwd_cross,wgrad,dgrad}_gemm: one LDS-tiled MFMA GEMM core
//    C[m][n] = sum_k A[m][k] B[n][k] (contraction index contiguous in both
//    operands, fp32 accumulation) with role-specific fused epilogues:
//      forward      y = relu(acc + b)                (Eq. 1, linear block body)
//      forward DCN  y = x0 * (acc + b) + x_l         (cross layer)
//      weight grad  dW partial slice, plus the bias gradient as row sums of
//                   the A operand (A = activation gradient, feature-major)
//      input grad   g = acc (+ g_out for a cross layer), then either the ReLU
//                   mask of the layer below or the cross-layer factor x0.
//    Every activation and activation gradient is produced in both a
//    row-major [M][N] and a feature-major [N][M] copy so that all three
//    GEMMs of a layer read K-contiguous operands with 16-byte loads.
//  * erase_head_bce: local head s = z w + c, sigmoid-BCE loss and its
//    gradient at z (the block's local objective, Section 2.1), with
//    deterministic per-workgroup partial sums.
//  * erase_adam: ordered reduction of the split partials, Adam update of the
//    fp32 master weights, and the bf16 GEMM copies of the new weights.
//  * erase_prologue: step counter increment and the feature-major copy of x.
//
// No float atomics anywhere: every reduction has a fixed order, so every
// schedule of the same step produces bit-identical results.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace erase {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// element conversions (bf16 is carried as uint16_t)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest, ties to even
  return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float ldf(const T* p);
template <> __device__ __forceinline__ float ldf<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ldf<uint16_t>(const uint16_t* p) { return bf2f(*p); }

template <typename T> __device__ __forceinline__ T cvt(float f);
template <> __device__ __forceinline__ float cvt<float>(float f) { return f; }
template <> __device__ __forceinline__ uint16_t cvt<uint16_t>(float f) { return f2bf(f); }

template <typename T> __device__ __forceinline__ float asf(T v);
template <> __device__ __forceinline__ float asf<float>(float v) { return v; }
template <> __device__ __forceinline__ float asf<uint16_t>(uint16_t v) { return bf2f(v); }

// Four consecutive elements of one feature-major row: one 8- or 16-byte store.
__device__ __forceinline__ void st4(uint16_t* p, const uint16_t v[4]) {
  uint2 w;
  w.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
  w.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
  *reinterpret_cast<uint2*>(p) = w;
}
__device__ __forceinline__ void st4(float* p, const float v[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ---------------------------------------------------------------------------
// GEMM core
// ---------------------------------------------------------------------------
template <typename T> struct GT;
// bf16: 16-byte chunk = 8 elements, k-step 64, v_mfma_f32_16x16x32_bf16
template <> struct GT<uint16_t> { static constexpr int KCH = 8, BK = 64, KMF = 32; };
// fp32: 16-byte chunk = 4 elements, k-step 32, v_mfma_f32_16x16x4_f32
template <> struct GT<float> { static constexpr int KCH = 4, BK = 32, KMF = 4; };

// One 16-byte chunk of row `row`, contraction elements [k, k+KCH), zero
// outside rows < nrows and k < kend.  Only in-range elements are read.
template <typename T>
__device__ __forceinline__ uint4 load_chunk(const T* P, int64_t ld, int row, int nrows, int k, int kend) {
  constexpr int KCH = GT<T>::KCH;
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (row < nrows && k < kend) {
    const T* p = P + (int64_t)row * ld + k;
    if (k + KCH <= kend) {
      v = *reinterpret_cast<const uint4*>(p);
    } else {
      T tmp[KCH];
#pragma unroll
      for (int e = 0; e < KCH; ++e) tmp[e] = (k + e < kend) ? p[e] : T(0);
      __builtin_memcpy(&v, tmp, 16);
    }
  }
  return v;
}

__device__ __forceinline__ float sum8_bf16(const uint4& a) {
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s += __uint_as_float(w[i] << 16);
    s += __uint_as_float(w[i] & 0xffff0000u);
  }
  return s;
}

template <typename T, int KIND>
__device__ __forceinline__ void epilogue4(const GemmDesc& g, const EpiParams& e, int mb, int n, const f32x4_t& acc,
                                          int z) {
  const int M = g.M;
  if constexpr (KIND == GK_FWD_RELU || KIND == GK_FWD_CROSS) {
    const float bn = e.bias[n];
    T* Y = static_cast<T*>(e.y);
    T o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = mb + q;
      float v = acc[q] + bn;
      if constexpr (KIND == GK_FWD_RELU) {
        v = v < 0.f ? 0.f : v;  // keeps NaN, like max(h, 0) on the host
      } else {
        if (m < M) {
          const float x0 = ldf(static_cast<const T*>(e.x0) + (int64_t)m * e.ldx0 + n);
          const float xl = ldf(static_cast<const T*>(e.xl) + (int64_t)m * e.ldxl + n);
          v = fmaf(x0, v, xl);
        }
      }
      o[q] = cvt<T>(v);
      if (m < M) Y[(int64_t)m * e.ldy + n] = o[q];
    }
    if (e.yt) {
      T* Yt = static_cast<T*>(e.yt) + (int64_t)n * e.ldyt;
      if (mb + 3 < M) {
        st4(Yt + mb, o);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (mb + q < M) Yt[mb + q] = o[q];
      }
    }
  } else if constexpr (KIND == GK_WGRAD) {
    float* P = e.part + (int64_t)z * e.pstride;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (mb + q < M) P[(int64_t)(mb + q) * e.ldp + n] = acc[q];
  } else {  // GK_DGRAD
    T d[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = mb + q;
      d[q] = T(0);
      if (m >= M) continue;
      float v = acc[q];
      if (e.res) v += ldf(static_cast<const T*>(e.res) + (int64_t)m * e.ldres + n);
      if (!e.below_cross) {
        const float mk = ldf(static_cast<const T*>(e.mask) + (int64_t)m * e.ldmask + n);
        d[q] = cvt<T>(mk > 0.f ? v : 0.f);
      } else {
        const T gq = cvt<T>(v);
        if (e.gout) static_cast<T*>(e.gout)[(int64_t)m * e.ldgout + n] = gq;
        const float x0 = ldf(static_cast<const T*>(e.x0) + (int64_t)m * e.ldx0 + n);
        d[q] = cvt<T>(asf(gq) * x0);
      }
      if (e.dmn) static_cast<T*>(e.dmn)[(int64_t)m * e.lddmn + n] = d[q];
    }
    T* Dt = static_cast<T*>(e.dnm) + (int64_t)n * e.lddnm;
    if (mb + 3 < M) {
      st4(Dt + mb, d);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (mb + q < M) Dt[mb + q] = d[q];
    }
  }
}

// Workgroup of 256 threads = 4 waves in a 2x2 arrangement; each wave owns a
// (BM/2) x (BN/2) sub-tile built from 16x16 MFMA tiles.  One LDS buffer per
// operand with register prefetch of the next k-step; LDS rows are padded by
// 16 bytes so the 16 rows read by one MFMA fragment hit distinct banks.
template <typename T, int BM, int BN, int KIND>
__device__ __forceinline__ void gemm_body(const GemmDesc& g, const EpiParams& e) {
  constexpr int BK = GT<T>::BK, KCH = GT<T>::KCH, KMF = GT<T>::KMF;
  constexpr int PITCH = BK + KCH;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
  constexpr int CPR = BK / KCH;
  constexpr int CA = BM * CPR / 256, CB = BN * CPR / 256;
  static_assert(CA * 256 == BM * CPR && CB * 256 == BN * CPR, "tile does not match 256 threads");
  __shared__ __attribute__((aligned(16))) T sA[BM * PITCH];
  __shared__ __attribute__((aligned(16))) T sB[BN * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int z = blockIdx.z;
  const int kbeg = z * g.kps;
  const int kend = min(g.K, kbeg + g.kps);
  const T* A = static_cast<const T*>(g.A);
  const T* B = static_cast<const T*>(g.B);

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const bool do_rows = (KIND == GK_WGRAD) && e.bpart != nullptr && blockIdx.y == 0 && wn == 0;
  float rs[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) rs[i] = 0.f;

  uint4 ra[CA], rb[CB];
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + i * 256;
      ra[i] = load_chunk<T>(A, g.lda, m0 + c / CPR, g.M, k0 + (c % CPR) * KCH, kend);
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * 256;
      rb[i] = load_chunk<T>(B, g.ldb, n0 + c / CPR, g.N, k0 + (c % CPR) * KCH, kend);
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + i * 256;
      *reinterpret_cast<uint4*>(&sA[(c / CPR) * PITCH + (c % CPR) * KCH]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * 256;
      *reinterpret_cast<uint4*>(&sB[(c / CPR) * PITCH + (c % CPR) * KCH]) = rb[i];
    }
  };
  auto compute = [&]() {
#pragma unroll
    for (int ks = 0; ks < BK; ks += KMF) {
      if constexpr (sizeof(T) == 2) {
        uint4 fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          fa[i] = *reinterpret_cast<const uint4*>(&sA[(wm * WM + i * 16 + (lane & 15)) * PITCH + ks + (lane >> 4) * 8]);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          fb[j] = *reinterpret_cast<const uint4*>(&sB[(wn * WN + j * 16 + (lane & 15)) * PITCH + ks + (lane >> 4) * 8]);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[i]),
                                                                __builtin_bit_cast(bf16x8_t, fb[j]), acc[i][j], 0, 0, 0);
        if (do_rows) {
#pragma unroll
          for (int i = 0; i < TM; ++i) rs[i] += sum8_bf16(fa[i]);
        }
      } else {
        float fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[i] = sA[(wm * WM + i * 16 + (lane & 15)) * PITCH + ks + (lane >> 4)];
#pragma unroll
        for (int j = 0; j < TN; ++j) fb[j] = sB[(wn * WN + j * 16 + (lane & 15)) * PITCH + ks + (lane >> 4)];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i], fb[j], acc[i][j], 0, 0, 0);
        if (do_rows) {
#pragma unroll
          for (int i = 0; i < TM; ++i) rs[i] += fa[i];
        }
      }
    }
  };

  if (nk > 0) {
    gload(kbeg);
    sstore();
  }
  __syncthreads();
  for (int it = 0; it < nk; ++it) {
    const bool more = it + 1 < nk;
    if (more) gload(kbeg + (it + 1) * BK);
    compute();
    __syncthreads();
    if (more) sstore();
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int mb = m0 + wm * WM + i * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * WN + j * 16 + (lane & 15);
      if (n < g.N) epilogue4<T, KIND>(g, e, mb, n, acc[i][j], z);
    }
  }
  if (do_rows) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      float s = rs[i];
      s += __shfl_xor(s, 16, 64);
      s += __shfl_xor(s, 32, 64);
      const int m = m0 + wm * WM + i * 16 + lane;
      if (lane < 16 && m < g.M) e.bpart[(int64_t)z * g.M + m] = s;
    }
  }
}

template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void erase_fwd_gemm(GemmDesc g, EpiParams e) {
  gemm_body<T, BM, BN, GK_FWD_RELU>(g, e);
}
template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void erase_fwd_cross_gemm(GemmDesc g, EpiParams e) {
  gemm_body<T, BM, BN, GK_FWD_CROSS>(g, e);
}
template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void erase_wgrad_gemm(GemmDesc g, EpiParams e) {
  gemm_body<T, BM, BN, GK_WGRAD>(g, e);
}
template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void erase_dgrad_gemm(GemmDesc g, EpiParams e) {
  gemm_body<T, BM, BN, GK_DGRAD>(g, e);
}

template <typename T, int BM, int BN>
static hipError_t launch_gemm_t(int kind, const GemmDesc& g, const EpiParams& e, hipStream_t s) {
  dim3 grid((g.M + BM - 1) / BM, (g.N + BN - 1) / BN, g.split), block(256);
  switch (kind) {
    case GK_FWD_RELU: hipLaunchKernelGGL((erase_fwd_gemm<T, BM, BN>), grid, block, 0, s, g, e); break;
    case GK_FWD_CROSS: hipLaunchKernelGGL((erase_fwd_cross_gemm<T, BM, BN>), grid, block, 0, s, g, e); break;
    case GK_WGRAD: hipLaunchKernelGGL((erase_wgrad_gemm<T, BM, BN>), grid, block, 0, s, g, e); break;
    case GK_DGRAD: hipLaunchKernelGGL((erase_dgrad_gemm<T, BM, BN>), grid, block, 0, s, g, e); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int bf16, int kind, const GemmDesc& g, const EpiParams& e, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.split <= 0) return hipErrorInvalidValue;
  if (bf16) {
    if (g.bm == 128 && g.bn == 128) return launch_gemm_t<uint16_t, 128, 128>(kind, g, e, s);
    if (g.bm == 128 && g.bn == 64) return launch_gemm_t<uint16_t, 128, 64>(kind, g, e, s);
    if (g.bm == 64 && g.bn == 128) return launch_gemm_t<uint16_t, 64, 128>(kind, g, e, s);
    if (g.bm == 64 && g.bn == 64) return launch_gemm_t<uint16_t, 64, 64>(kind, g, e, s);
  } else {
    if (g.bm == 64 && g.bn == 64) return launch_gemm_t<float, 64, 64>(kind, g, e, s);
  }
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// step prologue: t += 1 and xt[k][m] = x[m][k] through a 64x64 LDS tile
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void erase_prologue(PrologueArgs a) {
  __shared__ T tile[64][65];
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) a.t[0] = a.t[0] + 1;
  if (a.xt == nullptr) return;
  const T* X = static_cast<const T*>(a.x);
  T* XT = static_cast<T*>(a.xt);
  const int k0 = blockIdx.x * 64, m0 = blockIdx.y * 64;
  const int c = threadIdx.x & 63, r4 = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = r4 + 4 * i;
    const int m = m0 + r, k = k0 + c;
    tile[r][c] = (m < a.M && k < a.K) ? X[(int64_t)m * a.ldx + k] : T(0);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = r4 + 4 * i;  // k within tile
    const int k = k0 + r, m = m0 + c;
    if (k < a.K && m < a.M) XT[(int64_t)k * a.ldxt + m] = tile[c][r];
  }
}

hipError_t launch_prologue(int bf16, const PrologueArgs& a, hipStream_t s) {
  dim3 grid(a.xt ? (a.K + 63) / 64 : 1, a.xt ? (a.M + 63) / 64 : 1), block(256);
  if (bf16)
    hipLaunchKernelGGL(erase_prologue<uint16_t>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(erase_prologue<float>, grid, block, 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// local head + sigmoid-BCE + gradient at z, HEAD_ROWS rows per workgroup
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void erase_head_bce(HeadArgs a) {
  __shared__ float s_ds[HEAD_ROWS];
  __shared__ float s_loss[HEAD_ROWS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = blockIdx.x * HEAD_ROWS;
  const int rows = min(HEAD_ROWS, a.M - r0);
  const T* Z = static_cast<const T*>(a.z);
  const float c = a.c[0];

  // logits, per-row loss and dl/ds (16 rows per wave)
  for (int i = 0; i < HEAD_ROWS / 4; ++i) {
    const int rl = wave * (HEAD_ROWS / 4) + i;
    float part = 0.f;
    if (rl < rows) {
      const T* zr = Z + (int64_t)(r0 + rl) * a.ldz;
      for (int n = lane; n < a.N; n += 64) part = fmaf(ldf(zr + n), a.w[n], part);
    }
    part = wave_sum(part);
    if (lane == 0) {
      float ds = 0.f, l = 0.f;
      if (rl < rows) {
        const float s = part + c;
        const float yv = a.y[r0 + rl];
        const float en = __expf(-fabsf(s));
        const float sig = s >= 0.f ? 1.f / (1.f + en) : en / (1.f + en);
        ds = a.lam * (sig - yv) * a.inv_m;
        l = fmaxf(s, 0.f) - s * yv + log1pf(en);
      }
      s_ds[rl] = ds;
      s_loss[rl] = l;
    }
  }
  __syncthreads();

  // gradient at the pre-activation of the last (ReLU) layer, row-major
  if (a.dmn) {
    T* D = static_cast<T*>(a.dmn);
    for (int idx = tid; idx < rows * a.N; idx += 256) {
      const int rl = idx / a.N, n = idx - rl * a.N;
      const int64_t m = r0 + rl;
      const float zv = ldf(Z + m * a.ldz + n);
      D[m * a.lddmn + n] = cvt<T>(zv > 0.f ? s_ds[rl] * a.w[n] : 0.f);
    }
  }
  // ... and feature-major
  {
    T* D = static_cast<T*>(a.dnm);
    for (int idx = tid; idx < a.N * HEAD_ROWS; idx += 256) {
      const int n = idx / HEAD_ROWS, rl = idx - n * HEAD_ROWS;
      if (rl >= rows) continue;
      const int64_t m = r0 + rl;
      const float zv = ldf(Z + m * a.ldz + n);
      D[(int64_t)n * a.lddnm + m] = cvt<T>(zv > 0.f ? s_ds[rl] * a.w[n] : 0.f);
    }
  }
  // partial head gradients and loss of this workgroup's rows (fixed order)
  for (int n = tid; n < a.N; n += 256) {
    float acc = 0.f;
    for (int rl = 0; rl < rows; ++rl) acc = fmaf(ldf(Z + (int64_t)(r0 + rl) * a.ldz + n), s_ds[rl], acc);
    a.pdw[(int64_t)blockIdx.x * a.N + n] = acc;
  }
  if (tid == 0) {
    float sd = 0.f, sl = 0.f;
    for (int rl = 0; rl < rows; ++rl) {
      sd += s_ds[rl];
      sl += s_loss[rl];
    }
    a.pdc[blockIdx.x] = sd;
    a.ploss[blockIdx.x] = sl;
  }
}

hipError_t launch_head(int bf16, const HeadArgs& a, hipStream_t s) {
  dim3 grid((a.M + HEAD_ROWS - 1) / HEAD_ROWS), block(256);
  if (bf16)
    hipLaunchKernelGGL(erase_head_bce<uint16_t>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(erase_head_bce<float>, grid, block, 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Adam over all parameter segments of one block (ADAM_CHUNK elements per
// workgroup), with the ordered reduction of split partials fused in front
// and the GEMM copies of the updated weights written behind.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_seg(const AdamSeg* seg, int nseg, int64_t chunk) {
  int s = 0;
  while (s + 1 < nseg && seg[s + 1].chunk0 <= chunk) ++s;
  return s;
}

template <typename T>
__global__ __launch_bounds__(256) void erase_adam(AdamArgs a) {
  const int64_t chunk = blockIdx.x;
  const AdamSeg sg = a.seg[find_seg(a.seg, a.nseg, chunk)];
  const double t = (double)a.t[0];
  const float bc1 = (float)(1.0 - pow((double)a.beta1, t));
  const float bc2s = (float)sqrt(1.0 - pow((double)a.beta2, t));
  const float step = a.lr / bc1;
  const float b1 = a.beta1, b2 = a.beta2;
  const int n = sg.rows * sg.cols;
  const int base = (int)((chunk - sg.chunk0) * ADAM_CHUNK);
  T* SH = static_cast<T*>(sg.sh);
  T* SHT = static_cast<T*>(sg.sht);
#pragma unroll
  for (int q = 0; q < ADAM_CHUNK / 256; ++q) {
    const int i = base + q * 256 + (int)threadIdx.x;
    if (i >= n) break;
    const int r = i / sg.cols, c = i - r * sg.cols;
    const float* pp = sg.part + (int64_t)r * sg.ldpart + c;
    float g = 0.f;
    for (int zz = 0; zz < sg.nsplit; ++zz) g += pp[(int64_t)zz * sg.pstride];
    if (sg.g) sg.g[i] = g;
    const float m = fmaf(b1, sg.m[i], (1.f - b1) * g);
    const float v = fmaf(b2, sg.v[i], (1.f - b2) * g * g);
    const float p = sg.p[i] - step * m / (sqrtf(v) / bc2s + a.eps);
    sg.m[i] = m;
    sg.v[i] = v;
    sg.p[i] = p;
    if (SH) SH[(int64_t)r * sg.ldsh + c] = cvt<T>(p);
    if (SHT) SHT[(int64_t)c * sg.ldsht + r] = cvt<T>(p);
  }
  if (chunk == 0 && threadIdx.x == 0 && a.ploss) {
    float L = 0.f;
    for (int i = 0; i < a.nloss; ++i) L += a.ploss[i];
    L *= a.inv_m;
    a.loss_out[0] = L;
    if (!(fabsf(L) <= 3.4e38f)) a.status[0] = 1;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void erase_refresh(AdamArgs a) {
  const int64_t chunk = blockIdx.x;
  const AdamSeg sg = a.seg[find_seg(a.seg, a.nseg, chunk)];
  const int n = sg.rows * sg.cols;
  const int base = (int)((chunk - sg.chunk0) * ADAM_CHUNK);
  T* SH = static_cast<T*>(sg.sh);
  T* SHT = static_cast<T*>(sg.sht);
  for (int q = 0; q < ADAM_CHUNK / 256; ++q) {
    const int i = base + q * 256 + (int)threadIdx.x;
    if (i >= n) break;
    const int r = i / sg.cols, c = i - r * sg.cols;
    const float p = sg.p[i];
    if (SH) SH[(int64_t)r * sg.ldsh + c] = cvt<T>(p);
    if (SHT) SHT[(int64_t)c * sg.ldsht + r] = cvt<T>(p);
  }
}

hipError_t launch_adam(int bf16, const AdamArgs& a, hipStream_t s) {
  dim3 grid((unsigned)a.nchunks), block(256);
  if (bf16)
    hipLaunchKernelGGL(erase_adam<uint16_t>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(erase_adam<float>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_refresh(int bf16, const AdamArgs& a, hipStream_t s) {
  dim3 grid((unsigned)a.nchunks), block(256);
  if (bf16)
    hipLaunchKernelGGL(erase_refresh<uint16_t>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(erase_refresh<float>, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace erase
