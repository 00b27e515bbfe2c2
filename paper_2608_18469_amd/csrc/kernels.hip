// HIP kernels of the detached-block training step, written for gfx950
// (CDNA4: 64-wide wavefronts, MFMA matrix cores, 160 KB LDS per CU).
//
//  * erase_{fwd,fwd_cross,fwd_head,wgrad,dgrad}_gemm: one LDS-tiled MFMA
//    GEMM core with fp32 accumulation and role-specific fused epilogues:
//      forward      y = relu(acc + b)                (Eq. 1, linear block body)
//      forward DCN  y = x0 * (acc + b) + x_l         (cross layer)
//      forward+head the last layer with the local head and loss (Eq. 2)
//      weight grad  dW partial slice, plus the bias gradient as row sums of
//                   the A operand (the activation gradient)
//      input grad   g = acc (+ g_out for a cross layer), then either the ReLU
//                   mask of the layer below or the cross-layer factor x0.
//    Every activation and activation gradient exists once, row-major
//    [batch][features].  The forward and input-gradient GEMMs contract over
//    contiguous features; the weight gradient contracts over the batch, i.e.
//    over rows: its tiles are stored k-major in LDS and the MFMA operands
//    come from gfx950's transposing LDS reads (ds_read_b64_tr_b16).
//    erase_bwd_gemm runs a layer's weight- and input-gradient GEMMs in one
//    launch; the *_kg2 forward kernels split every k-step over two groups of
//    four waves (launches of at most one workgroup per CU).
//  * erase_head_bce: local head s = z w + c, sigmoid-BCE loss and its
//    gradient at z (the block's local objective, Section 2.1), with
//    deterministic per-workgroup partial sums.
//  * erase_adam: ordered reduction of the split partials, Adam update of the
//    fp32 master weights, and the bf16 GEMM copies of the new weights.
//  * erase_prologue: step counter increment, Adam factors, and the
//    zero-padded copy of x the GEMMs read.
//
// No float atomics anywhere: every reduction has a fixed order, so every
// schedule of the same step produces bit-identical results.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <type_traits>

#include "internal.h"

namespace erase {

#define ERASE_LAUNCH(KERNEL, GRID, BLOCK, SHMEM, STREAM, EV, ...)                                   \
  do {                                                                                             \
    if ((EV).e0 || (EV).e1)                                                                        \
      hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, (EV).e0, (EV).e1, 0, __VA_ARGS__); \
    else                                                                                           \
      hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__);                        \
  } while (0)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));  // 16-byte chunk in registers

// ---------------------------------------------------------------------------
// element conversions (bf16 is carried as uint16_t)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// gfx950 converts in hardware (v_cvt_pk_bf16_f32): round to nearest, ties to
// even, NaN stays NaN, no branch.
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

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

// Pointers read from device memory (not kernel arguments) are generic to the
// compiler; this marks them global so loads and stores use the global path.
template <typename T>
__device__ __forceinline__ __attribute__((address_space(1))) T* gmem(T* p) {
  return (__attribute__((address_space(1))) T*)p;
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

__device__ __forceinline__ float sum8_bf16(const u32x4_t& a) {
  const uint32_t w[4] = {a[0], a[1], a[2], a[3]};
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s += __uint_as_float(w[i] << 16);
    s += __uint_as_float(w[i] & 0xffff0000u);
  }
  return s;
}

// An MFMA operand fragment (8 consecutive contraction indices of one row) from
// a k-major bf16 LDS tile: two transposing 8-byte reads, rows p and p + 4*pitch.
typedef short s16x4_t __attribute__((ext_vector_type(4)));
template <typename T>
__device__ __forceinline__ u32x4_t tr_frag(const T* p, int pitch) {
  typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * pitch));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return u32x4_t{a.x, a.y, b.x, b.y};
}

// GELU in its tanh form, 0.5 u (1 + tanh(c (u + a u^3))) with c = sqrt(2/pi),
// a = 0.044715, and its derivative
// 0.5 (1 + t) + 0.5 u (1 - t^2) c (1 + 3 a u^2), t = tanh(c (u + a u^3)).
constexpr float kGeluC = 0.7978845608028654f, kGeluA = 0.044715f;
// tanh(y) = 1 - 2 / (exp(2y) + 1) with the hardware exp2 and reciprocal
// (absolute error about 1e-7; +-1 in the limits, where exp2 gives inf or 0)
__device__ __forceinline__ float tanh_hw(float y) {
  const float e = __builtin_amdgcn_exp2f(y * 2.8853900817779268f);  // 2 log2(e)
  return 1.f - 2.f * __builtin_amdgcn_rcpf(e + 1.f);
}
__device__ __forceinline__ float gelu_f(float u) {
  const float t = tanh_hw(kGeluC * fmaf(kGeluA * u * u, u, u));
  return 0.5f * u * (1.f + t);
}
__device__ __forceinline__ float gelu_grad_f(float u) {
  const float t = tanh_hw(kGeluC * fmaf(kGeluA * u * u, u, u));
  return 0.5f * (1.f + t) + 0.5f * u * (1.f - t * t) * kGeluC * fmaf(3.f * kGeluA, u * u, 1.f);
}

// Value of the fused epilogue at (m, n), m < M and n < N, in the output type.
template <typename T, int KIND>
__device__ __forceinline__ T epi_value(const EpiParams& e, int m, int n, float acc, float bn) {
  if constexpr (KIND == GK_FWD_RELU || KIND == GK_FWD_HEAD) {
    const float v = acc + bn;
    return cvt<T>(v < 0.f ? 0.f : v);  // keeps NaN, like max(h, 0) on the host
  } else if constexpr (KIND == GK_FWD_CROSS) {
    const float x0 = ldf(static_cast<const T*>(e.x0) + (int64_t)m * e.ldx0 + n);
    const float xl = ldf(static_cast<const T*>(e.xl) + (int64_t)m * e.ldxl + n);
    return cvt<T>(fmaf(x0, acc + bn, xl));
  } else if constexpr (KIND == GK_FWD_LIN) {
    float v = acc;
    if (e.res) v += ldf(static_cast<const T*>(e.res) + (int64_t)m * e.ldres + n);
    return cvt<T>(v);
  } else if constexpr (KIND == GK_FWD_GELU) {
    return cvt<T>(gelu_f(acc));
  } else if constexpr (KIND == GK_DGRAD_GELU) {
    return cvt<T>(acc * gelu_grad_f(ldf(static_cast<const T*>(e.mask) + (int64_t)m * e.ldmask + n)));
  } else if constexpr (KIND == GK_FWD_LOGITS) {
    return cvt<T>(acc);
  } else {  // GK_DGRAD
    float v = acc;
    if (e.res) v += ldf(static_cast<const T*>(e.res) + (int64_t)m * e.ldres + n);
    if (!e.below_cross) {
      if (!e.mask) return cvt<T>(v);
      const float mk = ldf(static_cast<const T*>(e.mask) + (int64_t)m * e.ldmask + n);
      return cvt<T>(mk > 0.f ? v : 0.f);
    }
    const T gq = cvt<T>(v);
    if (e.gout) static_cast<T*>(e.gout)[(int64_t)m * e.ldgout + n] = gq;
    const float x0 = ldf(static_cast<const T*>(e.x0) + (int64_t)m * e.ldx0 + n);
    return cvt<T>(asf(gq) * x0);
  }
}

// Workgroup of 256 threads = 4 waves in a 2x2 arrangement; each wave owns a
// (BM/2) x (BN/2) sub-tile of 16x16 MFMA tiles.  Pipeline: two LDS stages
// and two register sets, so the global loads of k-step it+3 are issued while
// k-step it is computed and land two compute phases later; one barrier per
// k-step.  Operands are zero-padded, so loads are never masked.  bf16 tiles are
// stored in LDS as unpadded 128-byte rows whose eight 16-byte chunks are
// permuted by chunk ^ (row & 7): on gfx950 a 16-byte LDS read is served 16
// lanes at a time over 64 banks (lane quads {0,3,5,6} and {1,2,4,7} of each
// half-wave together) and a 16-byte write 8 consecutive lanes at a time over
// 32 banks; with this permutation both the MFMA fragment reads (16 rows, four
// chunks) and the tile stores (one row per 8 lanes) touch every bank once.
// fp32 tiles keep a 16-byte row pad.
// The epilogue stages the output tile in LDS and writes it with 16-byte
// stores, row-major and (forward / input gradient) feature-major.
// XCD-aware tile order.  A launch's workgroup i runs on XCD (i + c) % 8 for
// some c, so the workgroups i = r (mod 8) share one XCD and its L2.
// xcd_linear() renumbers them so that each XCD owns one contiguous range of
// logical tiles; tile_from() walks logical tiles in groups of `group` M-tiles
// (M fastest inside a group, then N, then the next group; split-K slices
// last), so each range is a compact block of output tiles whose A and B rows
// are fetched into that XCD's L2 once and reused there.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_linear(int bid, int total) {
  const int q = total / kXcds, r = total % kXcds;
  const int x = bid % kXcds, loc = bid / kXcds;
  return x * q + min(x, r) + loc;
}
struct TileIdx {
  int m, n, z;
};
__device__ __forceinline__ TileIdx tile_from(int t, int gm, int gn, int group) {
  const int per = gm * gn;
  const int z = t / per;
  int u = t - z * per;
  const int gsz = group * gn;
  const int gi = u / gsz;
  const int mf = gi * group;
  const int gh = min(group, gm - mf);
  u -= gi * gsz;
  return {mf + u % gh, u / gh, z};
}

// One Adam update (PyTorch semantics: bias-corrected moments, eps outside
// the square root): step = lr / (1 - beta1^t), bc2s = sqrt(1 - beta2^t).
__device__ __forceinline__ void adam_elem(float& p, float& m, float& v, float g, float b1, float b2, float step,
                                          float bc2s, float eps) {
  m = fmaf(b1, m, (1.f - b1) * g);
  v = fmaf(b2, v, (1.f - b2) * g * g);
  p = p - step * m / (sqrtf(v) / bc2s + eps);
}

template <typename T, int BM, int BN, int KIND, int BKX = 0>
struct GemmSmem {
  static constexpr int BK = BKX ? BKX : GT<T>::BK, KCH = GT<T>::KCH, PITCH = sizeof(T) == 2 ? BK : BK + KCH;
  // weight gradient: k-major tiles [BK][BM] and [BK][BN] (fp32 rows padded by 16)
  static constexpr bool KMAJ = KIND == GK_WGRAD;
  static constexpr int PAD = sizeof(T) == 2 ? 0 : 16;
  static constexpr int STAGE = KMAJ ? BK * (BM + BN + 2 * PAD) : (BM + BN) * PITCH;
  using OT = typename std::conditional<KIND == GK_WGRAD, float, T>::type;
  static constexpr int MAIN = 2 * STAGE * (int)sizeof(T);
  // the logits epilogue stages the fp32 accumulators ([BM][BN + 4] floats)
  static constexpr int TILE = KIND == GK_FWD_LOGITS ? BM * (BN + 4) * 4
                                                    : BM * (BN + 16 / (int)sizeof(OT)) * (int)sizeof(OT);
  // fused head: hw[BN], labels[BM], ds[BM], loss[BM], dw[2][BN], c (fp32),
  // past both the main-loop stages and the output tile
  static constexpr int HOFF = MAIN > TILE ? MAIN : TILE;
  static constexpr int BYTES = HOFF + (KIND == GK_FWD_HEAD ? (3 * BN + 3 * BM + 4) * 4 : 0);
  // two k-groups: k-group 1's partial tile and row sums, one 64-float row
  // per accumulator register and wave, added by k-group 0 after the main loop
  static constexpr int RED2 = 4 * ((BM / 32) * (BN / 32) * 4 + BM / 32) * 64 * 4;
  static constexpr int BYTES_KG2 = BYTES > RED2 ? BYTES : RED2;
};

// KG k-groups of four waves (256 * KG threads): every k-group owns the whole
// output tile and computes it over its own 1/KG of each k-step (KG = 2 gives
// a one-workgroup-per-CU tile two waves per SIMD); the partial tiles are
// added through LDS after the main loop.
template <typename T, int BM, int BN, int KIND, int R = 2, int KG = 1, int BKX = 0>
__device__ __forceinline__ void gemm_body(const GemmDesc& g, const EpiParams& e, int bx, int by, int bz,
                                          char* smem) {
  constexpr int BK = BKX ? BKX : GT<T>::BK, KCH = GT<T>::KCH, KMF = GT<T>::KMF;
  constexpr int NT = 256 * KG;  // threads
  constexpr bool SWZ = sizeof(T) == 2;  // chunk-permuted rows (bf16) or padded rows (fp32)
  constexpr int PITCH = SWZ ? BK : BK + KCH;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
  constexpr int CPR = BK / KCH;
  constexpr int CA = BM * CPR / NT, CB = BN * CPR / NT;
  static_assert(CA * NT == BM * CPR && CB * NT == BN * CPR, "tile does not match the thread count");
  static_assert(KG == 1 || (KG == 2 && KIND != GK_FWD_HEAD && (BK / KG) % KMF == 0),
                "two k-groups: not with the fused head");
  // Operand layouts.  Forward and input gradient ("NT"): A [M][K] and B [N][K]
  // with the contraction contiguous; LDS tiles keep rows of BK elements.
  // Weight gradient (k-major): A [K][M] and B [K][N], i.e. activation
  // gradients and layer inputs in their row-major layout with the batch as
  // the contraction; LDS tiles are k-major, rows of BM (BN) elements, and
  // bf16 fragments come from pairs of transposing LDS reads.
  constexpr bool KMAJ = GemmSmem<T, BM, BN, KIND, BKX>::KMAJ;
  constexpr int PAD = GemmSmem<T, BM, BN, KIND, BKX>::PAD;
  constexpr int PA = BM + PAD, PB = BN + PAD;  // k-major row pitches
  constexpr int CPA = BM / KCH, CPB = BN / KCH;  // 16-byte chunks per k-major row
  constexpr int RPA = NT / CPA, RPB = NT / CPB;  // k-major rows per pass of the workgroup's threads
  static_assert(!KMAJ || (BK % RPA == 0 && BK % RPB == 0), "k-major tile does not match 256 threads");
  static_assert(!KMAJ || !SWZ || ((CPA == 8 || CPA == 16) && (CPB == 8 || CPB == 16)),
                "k-major chunk permutation: 8 or 16 chunks per row");
  constexpr int AREG = KMAJ ? BK * PA : BM * PITCH;  // elements of the A part of a stage
  constexpr int STAGE = GemmSmem<T, BM, BN, KIND, BKX>::STAGE;
  using OT = typename std::conditional<KIND == GK_WGRAD, float, T>::type;
  constexpr int OCH = 16 / (int)sizeof(OT);
  constexpr int OPITCH = BN + OCH;
  T* lds = reinterpret_cast<T*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = KG == 1 ? 0 : __builtin_amdgcn_readfirstlane(wave >> 2);  // k-group
  const int wm = (wave >> 1) & 1, wn = wave & 1;
  const int m0 = bx * BM, n0 = by * BN;
  const int z = bz;
  const int kbeg = z * g.kps;
  const int kend = min(g.K, kbeg + g.kps);
  const T* A = static_cast<const T*>(g.A);
  const T* B = static_cast<const T*>(g.B);

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if constexpr (KIND == GK_FWD_HEAD) {
    // head inputs into LDS now; their latency hides behind the main loop
    float* hs = reinterpret_cast<float*>(smem + GemmSmem<T, BM, BN, KIND, BKX>::HOFF);
    for (int n = tid; n < BN; n += 256) hs[n] = n < g.N ? e.hw[n] : 0.f;
    for (int r = tid; r < BM; r += 256) hs[BN + r] = m0 + r < g.M ? e.labels[m0 + r] : 0.f;
    if (tid == 0) hs[3 * BN + 3 * BM] = e.hc[0];
  }

  // forward biases: loaded now, their latency hides behind the main loop
  float bnv[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = n0 + wn * WN + j * 16 + (lane & 15);
    bnv[j] = 0.f;
    if constexpr (KIND == GK_FWD_RELU || KIND == GK_FWD_CROSS || KIND == GK_FWD_HEAD) bnv[j] = (n < g.N) ? e.bias[n] : 0.f;
  }

  // input gradient below a ReLU (bf16, tiles of at most 64 x 64): the
  // thread's mask values are loaded now, their latency hidden behind the
  // main loop (the contraction of these launches is short), two per register
  constexpr bool PFM = KIND == GK_DGRAD && sizeof(T) == 2 && TM * TN <= 4;
  const bool pfm = PFM && e.mask != nullptr && !e.below_cross && kg == 0;
  uint32_t mkp[PFM ? TM * TN * 2 : 1] = {};
  if constexpr (PFM) {
    const uint16_t* mk = static_cast<const uint16_t*>(e.mask);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          uint32_t w = 0;
          if (pfm) {
            const int n = n0 + wn * WN + j * 16 + (lane & 15);
#pragma unroll
            for (int q2 = 0; q2 < 2; ++q2) {
              const int m = m0 + wm * WM + i * 16 + (lane >> 4) * 4 + 2 * h + q2;
              if (m < g.M && n < g.N) w |= (uint32_t)mk[(int64_t)m * e.ldmask + n] << (16 * q2);
            }
          }
          mkp[(i * TN + j) * 2 + h] = w;
        }
  }

  // logits: the epilogue's store pass gives each row LTPR threads of 8
  // consecutive columns; the reference
  // logit of each of the thread's rows (in units of log2) is loaded now,
  // its latency hidden behind the main loop
  constexpr float kL2e = 1.4426950408889634f;
  constexpr int LTPR = BN / 8, LRPP = NT / LTPR, LPASS = BM / LRPP;  // threads per row, rows per pass, passes
  float xrl[KIND == GK_FWD_LOGITS ? LPASS : 1];
  if constexpr (KIND == GK_FWD_LOGITS) {
    static_assert(sizeof(T) == 2 && LPASS * LRPP == BM && LTPR <= 64, "logits: bf16, store pass matching the tile");
#pragma unroll
    for (int p = 0; p < LPASS; ++p) {
      const int m = m0 + tid / LTPR + p * LRPP;
      xrl[p] = m < g.M ? e.xref[m] * kL2e : 0.f;
    }
  }

  // fused Adam: the tile's parameters and moments are loaded now (they do not
  // depend on the gradient), so their HBM latency hides behind the main loop
  // fused Adam: the 64x64 two k-group weight gradient only (a block's first
  // layer); every other instantiation leaves these registers out
  constexpr bool FADAM = KIND == GK_WGRAD && KG == 2 && BM == 64 && BN == 64;
  typedef float f32x4a_t __attribute__((ext_vector_type(4), aligned(4)));
  typedef __attribute__((address_space(1))) f32x4a_t gvec;
  constexpr int AQ = BN / 4;                                                  // items of 4 columns per row
  constexpr int AIT = FADAM ? (BM * AQ + NT - 1) / NT : 1;  // items per thread
  f32x4a_t apv[AIT], amv[AIT], avv[AIT];
  bool afull[AIT];
  int64_t afi[AIT];
  if constexpr (FADAM) {
#pragma unroll
    for (int it = 0; it < AIT; ++it) {
      const int c = tid + it * NT;
      const int m = m0 + c / AQ, n = n0 + (c % AQ) * 4;
      afull[it] = e.ap != nullptr && c < BM * AQ && m < g.M && n + 4 <= g.N;
      afi[it] = (int64_t)m * g.N + n;
      if (afull[it]) {
        apv[it] = *reinterpret_cast<const gvec*>(gmem(e.ap) + afi[it]);
        amv[it] = *reinterpret_cast<const gvec*>(gmem(e.am) + afi[it]);
        avv[it] = *reinterpret_cast<const gvec*>(gmem(e.av) + afi[it]);
      }
    }
  }

  const bool do_rows = (KIND == GK_WGRAD) && e.bpart != nullptr && by == 0 && wn == 0;
  float rs[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) rs[i] = 0.f;

  // R register sets: set r holds k-steps r, r+R, r+2R, ...; the loads of a
  // k-step are issued R compute phases before it is stored to LDS.  Deeper
  // look-ahead (R = 3, 4) measured no faster on these shapes: the loop is
  // bound by the load and LDS paths, not by load latency.
  u32x4_t ra[R][CA], rb[R][CB];
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  // k-step j covers [kbeg + j*BK, kbeg + (j+1)*BK); loads past the last
  // k-step are clamped onto it (in bounds, never computed)
  const int klast = kbeg + (nk > 0 ? nk - 1 : 0) * BK;
  // per-thread tile chunks: address of the first, element strides between a
  // thread's chunks (ia, ib) and per contraction index (ka, kb), LDS offsets
  constexpr int RSTEP = NT / CPR;  // NT: tile rows between a thread's chunks
  static_assert(KMAJ || !SWZ || (CPR == 8 && RSTEP % 8 == 0), "chunk permutation assumes 8 chunks per row");
  // k-major rows r are stored with 16-byte chunk j at j ^ kperm(r): with it
  // the transposing fragment reads (32 lanes per pass over 64 banks) and the
  // tile stores are conflict-free (measured with the LDS bank counters)
  auto kperm = [](int r, int cpr) { return 2 * ((r >> 1) & 1) + 4 * ((r >> 3) & 1) + (cpr == 16 ? 8 * (r & 1) : 0); };
  const T* pa;
  const T* pb;
  int64_t ia, ib, ka, kb;
  int sofa, sofb, sia, sib;
  if constexpr (KMAJ) {
    const int ra_ = tid / CPA, ca_ = tid % CPA, rb_ = tid / CPB, cb_ = tid % CPB;
    pa = A + (int64_t)ra_ * g.lda + m0 + ca_ * KCH;
    pb = B + (int64_t)rb_ * g.ldb + n0 + cb_ * KCH;
    ia = (int64_t)RPA * g.lda;
    ib = (int64_t)RPB * g.ldb;
    ka = g.lda;
    kb = g.ldb;
    sofa = ra_ * PA + (SWZ ? (ca_ ^ kperm(ra_, CPA)) : ca_) * KCH;
    sofb = AREG + rb_ * PB + (SWZ ? (cb_ ^ kperm(rb_, CPB)) : cb_) * KCH;
    sia = RPA * PA;
    sib = RPB * PB;
  } else {
    const int srow = tid / CPR, sch = tid % CPR;
    pa = A + (int64_t)(m0 + srow) * g.lda + sch * KCH;
    pb = B + (int64_t)(n0 + srow) * g.ldb + sch * KCH;
    ia = (int64_t)RSTEP * g.lda;
    ib = (int64_t)RSTEP * g.ldb;
    ka = 1;
    kb = 1;
    sofa = srow * PITCH + (SWZ ? (sch ^ (srow & 7)) : sch) * KCH;
    sofb = BM * PITCH + sofa;
    sia = RSTEP * PITCH;
    sib = RSTEP * PITCH;
  }

  // Register sets are only ever indexed by compile-time constants (the loops
  // below are fully unrolled), so they stay in VGPRs.
  // Every operand is zero-padded (see GemmDesc): loads are never masked.
#define ERASE_GLOAD(SET, KSTEP)                                                                       \
  do {                                                                                                \
    const int64_t k0_ = min(kbeg + (KSTEP) * BK, klast);                                              \
    _Pragma("unroll") for (int i = 0; i < CA; ++i)                                                    \
        ra[SET][i] = *reinterpret_cast<const u32x4_t*>(pa + i * ia + k0_ * ka);                         \
    _Pragma("unroll") for (int i = 0; i < CB; ++i)                                                    \
        rb[SET][i] = *reinterpret_cast<const u32x4_t*>(pb + i * ib + k0_ * kb);                         \
  } while (0)
#define ERASE_SSTORE(SET, ST)                                                                         \
  do {                                                                                                \
    T* sa_ = lds + (ST) * STAGE;                                                                      \
    _Pragma("unroll") for (int i = 0; i < CA; ++i)                                                    \
        *reinterpret_cast<u32x4_t*>(sa_ + sofa + i * sia) = ra[SET][i];                                 \
    _Pragma("unroll") for (int i = 0; i < CB; ++i)                                                    \
        *reinterpret_cast<u32x4_t*>(sa_ + sofb + i * sib) = rb[SET][i];                                 \
  } while (0)

  // fragment offset within a 16-row slab; slab rows start at multiples of 16,
  // so a lane's row & 7 is lane & 7
  const int frow = (lane & 15) * PITCH + (SWZ ? 0 : (lane >> 4) * (KMF / 4));
  const int fch = (lane >> 4) ^ (lane & 7);  // bf16: permuted chunk of k-offset 0
  // k-major bf16 fragments: lane (g, q, c) = (lane >> 4, (lane & 15) >> 2,
  // lane & 3) reads 4 elements of row ks + 8g + q (then + 4) at column
  // 4c of its 16-column block; within each 16 lanes the transposing read
  // hands lane l element l & 3 of the chunks read by lanes 4q' + (l >> 2),
  // i.e. rows ks + 8g + q' of column l & 15: the MFMA operand layout.
  // The rows' permutation bits do not depend on ks or the half.
  const int tg = lane >> 4, tq = (lane & 15) >> 2, tc = lane & 3;
  const int trow = 8 * tg + tq;
  const int hpa = kperm(trow, CPA), hpb = kperm(trow, CPB);
  int foa[TM], fob[TN];  // element offsets of the lane's fragment chunks in a stage
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int col = wm * WM + i * 16;
    foa[i] = KMAJ ? (SWZ ? trow * PA + (((col >> 3) + (tc >> 1)) ^ hpa) * 8 + (tc & 1) * 4
                         : tg * PA + col + (lane & 15))
                  : 0;
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int col = wn * WN + j * 16;
    fob[j] = KMAJ ? AREG + (SWZ ? trow * PB + (((col >> 3) + (tc >> 1)) ^ hpb) * 8 + (tc & 1) * 4
                                : tg * PB + col + (lane & 15))
                  : 0;
  }
#define ERASE_COMPUTE(ST)                                                                             \
  do {                                                                                                \
    if constexpr (KMAJ) {                                                                             \
      const T* st_ = lds + (ST) * STAGE;                                                              \
      _Pragma("unroll") for (int kk_ = 0; kk_ < BK / KG; kk_ += KMF) {                                \
        const int ks = kg * (BK / KG) + kk_; /* this k-group's part of the k-step */                   \
        if constexpr (sizeof(T) == 2) {                                                               \
          u32x4_t fa[TM], fb[TN];                                                                       \
          _Pragma("unroll") for (int i = 0; i < TM; ++i) fa[i] = tr_frag(st_ + foa[i] + ks * PA, PA);  \
          _Pragma("unroll") for (int j = 0; j < TN; ++j) fb[j] = tr_frag(st_ + fob[j] + ks * PB, PB);  \
          _Pragma("unroll") for (int i = 0; i < TM; ++i)                                              \
          _Pragma("unroll") for (int j = 0; j < TN; ++j)                                              \
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                                    \
                  __builtin_bit_cast(bf16x8_t, fa[i]), __builtin_bit_cast(bf16x8_t, fb[j]), acc[i][j], 0, 0, 0); \
          if (do_rows) {                                                                              \
            _Pragma("unroll") for (int i = 0; i < TM; ++i) rs[i] += sum8_bf16(fa[i]);                 \
          }                                                                                           \
        } else {                                                                                      \
          float fa[TM], fb[TN];                                                                       \
          _Pragma("unroll") for (int i = 0; i < TM; ++i) fa[i] = asf(st_[foa[i] + ks * PA]);          \
          _Pragma("unroll") for (int j = 0; j < TN; ++j) fb[j] = asf(st_[fob[j] + ks * PB]);          \
          _Pragma("unroll") for (int i = 0; i < TM; ++i)                                              \
          _Pragma("unroll") for (int j = 0; j < TN; ++j)                                              \
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i], fb[j], acc[i][j], 0, 0, 0);     \
          if (do_rows) {                                                                              \
            _Pragma("unroll") for (int i = 0; i < TM; ++i) rs[i] += fa[i];                            \
          }                                                                                           \
        }                                                                                             \
      }                                                                                               \
      break;                                                                                          \
    }                                                                                                 \
    const T* sa_ = lds + (ST) * STAGE + wm * WM * PITCH + frow;                                       \
    const T* sb_ = lds + (ST) * STAGE + BM * PITCH + wn * WN * PITCH + frow;                          \
    _Pragma("unroll") for (int kk_ = 0; kk_ < BK / KG; kk_ += KMF) {                                  \
      const int ks = kg * (BK / KG) + kk_; /* this k-group's part of the k-step */                     \
      if constexpr (sizeof(T) == 2) {                                                                 \
        const int ko_ = (fch ^ (ks / KCH)) * KCH;                                                     \
        u32x4_t fa[TM], fb[TN];                                                                         \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                                \
            fa[i] = *reinterpret_cast<const u32x4_t*>(sa_ + i * 16 * PITCH + ko_);                      \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                                \
            fb[j] = *reinterpret_cast<const u32x4_t*>(sb_ + j * 16 * PITCH + ko_);                      \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                                \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                                \
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                                      \
                __builtin_bit_cast(bf16x8_t, fa[i]), __builtin_bit_cast(bf16x8_t, fb[j]), acc[i][j], 0, 0, 0); \
        if (do_rows) {                                                                                \
          _Pragma("unroll") for (int i = 0; i < TM; ++i) rs[i] += sum8_bf16(fa[i]);                   \
        }                                                                                             \
      } else {                                                                                        \
        float fa[TM], fb[TN];                                                                         \
        _Pragma("unroll") for (int i = 0; i < TM; ++i) fa[i] = asf(sa_[i * 16 * PITCH + ks]);         \
        _Pragma("unroll") for (int j = 0; j < TN; ++j) fb[j] = asf(sb_[j * 16 * PITCH + ks]);         \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                                \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                                \
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i], fb[j], acc[i][j], 0, 0, 0);       \
        if (do_rows) {                                                                                \
          _Pragma("unroll") for (int i = 0; i < TM; ++i) rs[i] += fa[i];                              \
        }                                                                                             \
      }                                                                                               \
    }                                                                                                 \
  } while (0)

  // prologue: set r <- k-step r; stage 0 <- k-step 0; set 0 <- k-step R
  if (nk > 0) {
#pragma unroll
    for (int r = 0; r < R; ++r) ERASE_GLOAD(r, r);
    ERASE_SSTORE(0, 0);
    ERASE_GLOAD(0, R);
  }
  __syncthreads();
  // phase j: compute k-step j from stage j % 2, store k-step j+1 (set
  // (j+1) % R) into the other stage, refill that set with k-step j+1+R; one
  // barrier per phase.  The last phase ends with a barrier, so the epilogue
  // may reuse the LDS.
  constexpr int U = (R % 2 == 0) ? R : 2 * R;  // phases per unrolled round
  // Main loop: rounds of U phases whose loads are all real, with no branch
  // inside, so the waits before each LDS store count exactly the loads that
  // may stay in flight (behind a branch the compiler waits for all of them).
  // Tail: the last phases, straight-line, loading and staging only real
  // k-steps, so no load is left in flight for the epilogue to wait on.
  int base = 0;
  for (; base + U + R < nk; base += U) {
#pragma unroll
    for (int p = 0; p < U; ++p) {
      ERASE_COMPUTE(p % 2);
      ERASE_SSTORE((p + 1) % R, (p + 1) % 2);
      ERASE_GLOAD((p + 1) % R, base + p + 1 + R);
      __syncthreads();
    }
  }
#pragma unroll
  for (int p = 0; p < U + R + 1; ++p) {
    const int j = base + p;
    if (j < nk) {
      ERASE_COMPUTE(p % 2);
      if (j + 1 < nk) ERASE_SSTORE((p + 1) % R, (p + 1) % 2);
      if (j + 1 + R < nk) ERASE_GLOAD((p + 1) % R, j + 1 + R);
      __syncthreads();
    }
  }
#undef ERASE_GLOAD
#undef ERASE_SSTORE
#undef ERASE_COMPUTE

  if constexpr (KG == 2) {
    // k-group 1's partial tile (and bias row sums) into the (now free) stage
    // memory, one 64-float row per accumulator register and wave; k-group 0
    // adds them
    float* red = reinterpret_cast<float*>(smem);
    static_assert(4 * (TM * TN * 4 + TM) * 64 * 4 <= GemmSmem<T, BM, BN, KIND, BKX>::BYTES_KG2, "reduction buffer");
    const int sw = wave & 3;
    float* rrs = red + 4 * TM * TN * 4 * 64;
    if (kg == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) red[(((sw * TM + i) * TN + j) * 4 + q) * 64 + lane] = acc[i][j][q];
      if (do_rows) {
#pragma unroll
        for (int i = 0; i < TM; ++i) rrs[(sw * TM + i) * 64 + lane] = rs[i];
      }
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[i][j][q] += red[(((sw * TM + i) * TN + j) * 4 + q) * 64 + lane];
      if (do_rows) {
#pragma unroll
        for (int i = 0; i < TM; ++i) rs[i] += rrs[(sw * TM + i) * 64 + lane];
      }
    }
    __syncthreads();
  }

  if (do_rows && kg == 0) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      float sr = rs[i];
      sr += __shfl_xor(sr, 16, 64);
      sr += __shfl_xor(sr, 32, 64);
      const int m = m0 + wm * WM + i * 16 + lane;
      if (lane < 16 && m < g.M) {
        if constexpr (FADAM) {
          if (e.bp) {
            // fused Adam of the bias: this tile holds its rows' whole gradient
            float p = e.bp[m], mo = e.bm[m], v = e.bv[m];
            adam_elem(p, mo, v, sr, e.b1, e.b2, e.hyper[0], e.hyper[1], e.eps);
            if (e.bg) e.bg[m] = sr;
            e.bm[m] = mo;
            e.bv[m] = v;
            e.bp[m] = p;
            continue;
          }
        }
        e.bpart[(int64_t)z * g.M + m] = sr;
      }
    }
  }

  // epilogue: values -> LDS tile [BM][OPITCH] -> 16-byte row-major stores.
  OT* sc = reinterpret_cast<OT*>(smem);
  const int M = g.M, N = g.N;
  OT* omn;
  int64_t ldmn;
  if constexpr (KIND == GK_WGRAD) {
    omn = e.part + (int64_t)z * e.pstride;
    ldmn = e.ldp;
  } else if constexpr (KIND == GK_DGRAD || KIND == GK_DGRAD_GELU) {
    omn = static_cast<OT*>(e.dmn);
    ldmn = e.lddmn;
  } else {
    omn = static_cast<OT*>(e.y);
    ldmn = e.ldy;
  }
  // pass 1 (every load of the epilogue): values into the LDS tile and back
  // into the accumulators; pass 2 (stores only): the row-major tile.
  // Keeping loads and stores apart avoids waits on the stores (on gfx9 the
  // load counter also counts stores).  With two k-groups, k-group 0 holds
  // the sums.
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    if (kg != 0) break;
    const int nl = wn * WN + j * 16 + (lane & 15);
    const int n = n0 + nl;
    const float bn = bnv[j];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int ml = wm * WM + i * 16 + (lane >> 4) * 4 + q;
        const int m = m0 + ml;
        if constexpr (KIND == GK_FWD_LOGITS) {
          // the fp32 accumulators as they are; the store pass exponentiates
          reinterpret_cast<float*>(smem)[ml * (BN + 4) + nl] = acc[i][j][q];
          continue;
        }
        OT v;
        if constexpr (KIND == GK_WGRAD) {
          v = acc[i][j][q];
        } else {
          if (PFM && pfm) {
            // epi_value's masked input gradient with the prefetched mask
            float a = acc[i][j][q];
            if (e.res && m < M && n < N) a += ldf(static_cast<const T*>(e.res) + (int64_t)m * e.ldres + n);
            const uint32_t mb = (mkp[PFM ? (i * TN + j) * 2 + (q >> 1) : 0] >> (16 * (q & 1))) & 0xffffu;
            v = (m < M && n < N) ? cvt<T>(__uint_as_float(mb << 16) > 0.f ? a : 0.f) : OT(0);
          } else {
            v = (m < M && n < N) ? epi_value<T, KIND>(e, m, n, acc[i][j][q], bn) : OT(0);
          }
          if constexpr (KIND != GK_FWD_GELU) acc[i][j][q] = asf(v);  // GELU keeps the pre-activation
        }
        sc[ml * OPITCH + nl] = v;
      }
    }
  }
  __syncthreads();
  bool store_tile = omn != nullptr;
  // fused Adam (two k-group weight gradients only) reads the LDS tile instead
  if constexpr (FADAM) store_tile = store_tile && e.ap == nullptr;
  // logits: the store pass below exponentiates as it stores
  if constexpr (KIND == GK_FWD_LOGITS) store_tile = false;
  if (store_tile) {
    constexpr int CPRO = BN / OCH;
    for (int c = tid; c < BM * CPRO; c += NT) {
      const int ml = c / CPRO, nl = (c % CPRO) * OCH;
      const int m = m0 + ml, n = n0 + nl;
      if (m >= M || n >= N) continue;
      const OT* src = &sc[ml * OPITCH + nl];
      OT* dst = omn + (int64_t)m * ldmn + n;
      if (n + OCH <= N) {
        *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
      } else {
        for (int q = 0; q < OCH && n + q < N; ++q) dst[q] = src[q];
      }
    }
  }

  if constexpr (KIND == GK_FWD_GELU) {
    // the pre-activation u = acc into gout, through the same LDS tile
    if (e.gout) {
      __syncthreads();
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int nl = wn * WN + j * 16 + (lane & 15);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int ml = wm * WM + i * 16 + (lane >> 4) * 4 + q;
            sc[ml * OPITCH + nl] = (m0 + ml < M && n0 + nl < N) ? cvt<T>(acc[i][j][q]) : OT(0);
          }
      }
      __syncthreads();
      constexpr int CPRO = BN / OCH;
      for (int c = tid; c < BM * CPRO; c += NT) {
        const int ml = c / CPRO, nl = (c % CPRO) * OCH;
        const int m = m0 + ml, n = n0 + nl;
        if (m >= M || n >= N) continue;
        const OT* src = &sc[ml * OPITCH + nl];
        OT* dst = static_cast<OT*>(e.gout) + (int64_t)m * e.ldgout + n;
        if (n + OCH <= N) {
          *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
        } else {
          for (int q = 0; q < OCH && n + q < N; ++q) dst[q] = src[q];
        }
      }
    }
  }

  if constexpr (KIND == GK_FWD_LOGITS) {
    // Store pass: y = exp(acc - xref) rounded to bf16 (pairs converted by
    // one instruction), one 16-byte store of 8 consecutive columns per
    // thread and row, and the row's sum of the stored values: the thread's
    // 8 in column order, then a butterfly over the row's LTPR lanes (the
    // same sum in every lane), so the order is fixed.  Columns past N are
    // neither stored nor summed (only the last column tile has any).
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const float* scf = reinterpret_cast<const float*>(smem);
    uint16_t* Y = static_cast<uint16_t*>(e.y);
    const int tq = tid % LTPR, r0 = tid / LTPR, c0 = 8 * tq;
    const bool full = n0 + BN <= N;
#pragma unroll
    for (int p = 0; p < LPASS; ++p) {
      const int ml = r0 + p * LRPP, m = m0 + ml, n = n0 + c0;
      const f32x4_t xa = *reinterpret_cast<const f32x4_t*>(&scf[ml * (BN + 4) + c0]);
      const f32x4_t xb = *reinterpret_cast<const f32x4_t*>(&scf[ml * (BN + 4) + c0 + 4]);
      float ev[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        ev[k] = __builtin_amdgcn_exp2f(fmaf(xa[k], kL2e, -xrl[p]));
        ev[4 + k] = __builtin_amdgcn_exp2f(fmaf(xb[k], kL2e, -xrl[p]));
      }
      if (!full) {
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (n + k >= N) ev[k] = 0.f;
      }
      u32x4_t o;
      float se = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        o[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{ev[2 * k], ev[2 * k + 1]}), bf16x2_t));
        se += __uint_as_float(o[k] << 16);
        se += __uint_as_float(o[k] & 0xffff0000u);
      }
      if (m < M) {
        uint16_t* dst = Y + (int64_t)m * e.ldy + n;
        if (full || n + 8 <= N) {
          *reinterpret_cast<u32x4_t*>(dst) = o;
        } else {
          for (int k = 0; k < 8 && n + k < N; ++k) dst[k] = (uint16_t)(k & 1 ? o[k / 2] >> 16 : o[k / 2] & 0xffffu);
        }
      }
#pragma unroll
      for (int q = 1; q < LTPR; q <<= 1) se += __shfl_xor(se, q, 64);
      if (tq == 0 && m < M) e.lstat[(int64_t)m * e.ldlstat + by] = se;
    }
  }

  // Only the two k-group kernels take the fused update: its per-thread item
  // arrays would otherwise hold a 128x128 tile's registers in every
  // weight-gradient instantiation (one wave per SIMD).
  if constexpr (FADAM) {
    if (e.ap) {
      // Fused Adam: the LDS tile holds this tile's finished gradient (the
      // contraction is not split).  Items of 4 consecutive columns of one
      // row (16-byte accesses at 4-byte alignment: parameter rows start
      // anywhere), whose parameters and moments were loaded before the main
      // loop; a row's ragged end goes element by element.
      const float step = e.hyper[0], bc2s = e.hyper[1];
      constexpr int Q = AQ, IT = AIT;
      f32x4_t gv[IT];
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int c = tid + it * NT;
        if (afull[it]) gv[it] = *reinterpret_cast<const f32x4_t*>(&sc[(c / Q) * OPITCH + (c % Q) * 4]);
      }
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int c = tid + it * NT;
        const int ml = c / Q, nl = (c % Q) * 4;
        const int m = m0 + ml, n = n0 + nl;
        if (afull[it]) {
          float pp[4], mm[4], vq[4];
          T o[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            pp[k] = apv[it][k];
            mm[k] = amv[it][k];
            vq[k] = avv[it][k];
            adam_elem(pp[k], mm[k], vq[k], gv[it][k], e.b1, e.b2, step, bc2s, e.eps);
            o[k] = cvt<T>(pp[k]);
          }
          if (e.ag) *reinterpret_cast<gvec*>(gmem(e.ag) + afi[it]) = f32x4a_t{gv[it][0], gv[it][1], gv[it][2], gv[it][3]};
          *reinterpret_cast<gvec*>(gmem(e.am) + afi[it]) = f32x4a_t{mm[0], mm[1], mm[2], mm[3]};
          *reinterpret_cast<gvec*>(gmem(e.av) + afi[it]) = f32x4a_t{vq[0], vq[1], vq[2], vq[3]};
          *reinterpret_cast<gvec*>(gmem(e.ap) + afi[it]) = f32x4a_t{pp[0], pp[1], pp[2], pp[3]};
          st4(static_cast<T*>(e.ash) + (int64_t)m * e.ldash + n, o);  // copy rows: 64-element multiples
        } else if (c < BM * Q && m < M && n < N) {
          for (int k = 0; k < N - n && k < 4; ++k) {
            const float gk = sc[ml * OPITCH + nl + k];
            float pp = e.ap[afi[it] + k], mm = e.am[afi[it] + k], vq = e.av[afi[it] + k];
            adam_elem(pp, mm, vq, gk, e.b1, e.b2, step, bc2s, e.eps);
            if (e.ag) e.ag[afi[it] + k] = gk;
            e.am[afi[it] + k] = mm;
            e.av[afi[it] + k] = vq;
            e.ap[afi[it] + k] = pp;
            static_cast<T*>(e.ash)[(int64_t)m * e.ldash + n + k] = cvt<T>(pp);
          }
        }
      }
    }
  }

  if constexpr (KIND == GK_FWD_HEAD) {
    // Fused local head (Section 2.1, Eq. 2).  The tile holds complete rows
    // of the block output z (N <= BN, one tile column, n0 = 0):
    //   s_m = sum_n z_mn w_n + c,  loss_m = max(s,0) - s y_m + log1p(e^-|s|),
    //   ds_m = lam (sigmoid(s_m) - y_m) / M,  dz_mn = ds_m w_n [z_mn > 0]
    // in both layouts, and this M-tile's partials dw_n = sum_m z_mn ds_m,
    // dc = sum_m ds_m and sum_m loss_m, every sum in a fixed order.
    float* s_w = reinterpret_cast<float*>(smem + GemmSmem<T, BM, BN, KIND, BKX>::HOFF);
    float* s_y = s_w + BN;
    float* s_ds = s_y + BM;
    float* s_l = s_ds + BM;
    float* s_dw = s_l + BM;  // [2][BN]: per row-half of the waves
    const float hc = s_dw[2 * BN];
    constexpr int KC = OCH;
    {  // logits: TPR lanes per row over contiguous column slices, fixed butterfly
      constexpr int TPR = 256 / BM;
      static_assert(TPR * BM == 256 && (TPR & (TPR - 1)) == 0 && TPR <= 64, "head rows do not match 256 threads");
      constexpr int CPT = BN / TPR;
      const int r = tid / TPR, jj = tid % TPR;
      float part = 0.f;
#pragma unroll 8
      for (int q = 0; q < CPT; ++q) part = fmaf(asf(sc[r * OPITCH + jj * CPT + q]), s_w[jj * CPT + q], part);
      for (int off = 1; off < TPR; off <<= 1) part += __shfl_xor(part, off, 64);
      if (jj == 0) {
        float ds = 0.f, l = 0.f;
        if (m0 + r < M) {
          const float sv = part + hc;
          const float yv = s_y[r];
          const float en = __expf(-fabsf(sv));
          const float sig = sv >= 0.f ? 1.f / (1.f + en) : en / (1.f + en);
          ds = e.lam * (sig - yv) * e.inv_m;
          l = fmaxf(sv, 0.f) - sv * yv + log1pf(en);
        }
        s_ds[r] = ds;
        s_l[r] = l;
      }
    }
    __syncthreads();
    // this wave's column sums of z ds, from the accumulators
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nl = wn * WN + j * 16 + (lane & 15);
      float dwp = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int ml0 = wm * WM + i * 16 + (lane >> 4) * 4;
#pragma unroll
        for (int q = 0; q < 4; ++q) dwp = fmaf(acc[i][j][q], s_ds[ml0 + q], dwp);  // z as stored (0 outside M x N)
      }
      // lanes l, l^16, l^32, l^48 hold the same column (rows 4 apart)
      dwp += __shfl_xor(dwp, 16, 64);
      dwp += __shfl_xor(dwp, 32, 64);
      if (lane < 16) s_dw[wm * BN + nl] = dwp;
    }
    // dz row-major (input gradient of the last layer's GEMM; nullable)
    if (e.dmn) {
      constexpr int CPRO = BN / KC;
      for (int c = tid; c < BM * CPRO; c += 256) {
        const int r = c / CPRO, nl = (c % CPRO) * KC;
        const int m = m0 + r, n = n0 + nl;
        if (m >= M || n >= N) continue;
        const float ds = s_ds[r];
        OT o[KC];
#pragma unroll
        for (int q = 0; q < KC; ++q) {
          const float zq = asf(sc[r * OPITCH + nl + q]);
          o[q] = cvt<T>(zq > 0.f ? ds * s_w[nl + q] : 0.f);
        }
        OT* dst = static_cast<OT*>(e.dmn) + (int64_t)m * e.lddmn + n;
        if (n + KC <= N) {
          uint4 v;
          __builtin_memcpy(&v, o, 16);
          *reinterpret_cast<uint4*>(dst) = v;
        } else {
#pragma unroll
          for (int q = 0; q < KC; ++q)
            if (n + q < N) dst[q] = o[q];
        }
      }
    }
    __syncthreads();
    for (int n = tid; n < N; n += 256) e.pdw[(int64_t)bx * N + n] = s_dw[n] + s_dw[BN + n];
    if (tid < 64) {
      float d = 0.f, l = 0.f;
      for (int r = tid; r < BM; r += 64) {
        d += s_ds[r];
        l += s_l[r];
      }
      d = wave_sum(d);
      l = wave_sum(l);
      if (tid == 0) {
        e.pdc[bx] = d;
        e.ploss[bx] = l;
      }
    }
  }
}

#define ERASE_GEMM_KERNEL(NAME, KIND)                                                    \
  template <typename T, int BM, int BN>                                                  \
  __global__ __launch_bounds__(256) void NAME(GemmDesc g, EpiParams e) {                 \
    __shared__ __attribute__((aligned(16))) char smem[GemmSmem<T, BM, BN, KIND>::BYTES]; \
    const int gm = (g.M + BM - 1) / BM, gn = (g.N + BN - 1) / BN;                        \
    const TileIdx ti = tile_from(xcd_linear(blockIdx.x, gridDim.x), gm, gn, g.group);   \
    gemm_body<T, BM, BN, KIND>(g, e, ti.m, ti.n, ti.z, smem);                            \
  }
ERASE_GEMM_KERNEL(erase_fwd_gemm, GK_FWD_RELU)
ERASE_GEMM_KERNEL(erase_fwd_cross_gemm, GK_FWD_CROSS)
ERASE_GEMM_KERNEL(erase_wgrad_gemm, GK_WGRAD)
ERASE_GEMM_KERNEL(erase_dgrad_gemm, GK_DGRAD)
ERASE_GEMM_KERNEL(erase_fwd_head_gemm, GK_FWD_HEAD)
ERASE_GEMM_KERNEL(erase_fwd_lin_gemm, GK_FWD_LIN)
ERASE_GEMM_KERNEL(erase_fwd_gelu_gemm, GK_FWD_GELU)
ERASE_GEMM_KERNEL(erase_dgrad_gelu_gemm, GK_DGRAD_GELU)
ERASE_GEMM_KERNEL(erase_fwd_logits_gemm, GK_FWD_LOGITS)
#undef ERASE_GEMM_KERNEL

// Two k-groups of four waves (512 threads): forward tiles of launches with at
// most one workgroup per CU, which then run two waves per SIMD.
#define ERASE_GEMM_KERNEL_KG2(NAME, KIND, BKX)                                                \
  template <typename T, int BM, int BN>                                                       \
  __global__ __launch_bounds__(512) void NAME(GemmDesc g, EpiParams e) {                      \
    constexpr int BKK = sizeof(T) == 2 ? BKX : 0;                                            \
    __shared__ __attribute__((aligned(16))) char smem[GemmSmem<T, BM, BN, KIND, BKK>::BYTES_KG2]; \
    const int gm = (g.M + BM - 1) / BM, gn = (g.N + BN - 1) / BN;                             \
    const TileIdx ti = tile_from(xcd_linear(blockIdx.x, gridDim.x), gm, gn, g.group);        \
    gemm_body<T, BM, BN, KIND, 2, 2, BKK>(g, e, ti.m, ti.n, ti.z, smem);                      \
  }
ERASE_GEMM_KERNEL_KG2(erase_fwd_gemm_kg2, GK_FWD_RELU, 0)
ERASE_GEMM_KERNEL_KG2(erase_fwd_cross_gemm_kg2, GK_FWD_CROSS, 0)
// the weight gradient: k-steps of 128 batch rows (bf16), two MFMA k-steps
// per k-group between barriers
ERASE_GEMM_KERNEL_KG2(erase_wgrad_gemm_kg2, GK_WGRAD, 128)
#undef ERASE_GEMM_KERNEL_KG2

// One launch for both backward GEMMs of a layer (they read the same
// activation gradient and are independent): workgroups [0, nw) compute the
// weight-gradient tiles and slices (the longer contractions, so they start
// first), the rest the input-gradient tiles.
template <typename T, int BM, int BN, int KG>
__device__ __forceinline__ void bwd_pair(const GemmDesc& gd, const EpiParams& ed, const GemmDesc& gw,
                                         const EpiParams& ew, int nw, char* smem) {
  // each GEMM is renumbered on its own (workgroups b and b + 8 still share an
  // XCD after subtracting nw), so both spread evenly over the XCDs
  const int b = blockIdx.x;
  if (b < nw) {
    const TileIdx ti = tile_from(xcd_linear(b, nw), (gw.M + BM - 1) / BM, (gw.N + BN - 1) / BN, gw.group);
    gemm_body<T, BM, BN, GK_WGRAD, 2, KG>(gw, ew, ti.m, ti.n, ti.z, smem);
  } else {
    const int nd = gridDim.x - nw;
    const TileIdx ti = tile_from(xcd_linear(b - nw, nd), (gd.M + BM - 1) / BM, (gd.N + BN - 1) / BN, gd.group);
    gemm_body<T, BM, BN, GK_DGRAD, 2, KG>(gd, ed, ti.m, ti.n, 0, smem);
  }
}

template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void erase_bwd_gemm(GemmDesc gd, EpiParams ed, GemmDesc gw, EpiParams ew, int nw) {
  constexpr int SD = GemmSmem<T, BM, BN, GK_DGRAD>::BYTES, SW = GemmSmem<T, BM, BN, GK_WGRAD>::BYTES;
  __shared__ __attribute__((aligned(16))) char smem[SD > SW ? SD : SW];
  bwd_pair<T, BM, BN, 1>(gd, ed, gw, ew, nw, smem);
}

// The same pair with 512-thread workgroups: two k-groups of four waves, each
// over half of every k-step of the whole tile, so every SIMD runs two waves
// of one tile (the large 128x128 tiles, one workgroup per CU).
template <typename T, int BM, int BN>
__global__ __launch_bounds__(512) void erase_bwd_gemm_kg2(GemmDesc gd, EpiParams ed, GemmDesc gw, EpiParams ew,
                                                          int nw) {
  constexpr int SD = GemmSmem<T, BM, BN, GK_DGRAD>::BYTES_KG2, SW = GemmSmem<T, BM, BN, GK_WGRAD>::BYTES_KG2;
  __shared__ __attribute__((aligned(16))) char smem[SD > SW ? SD : SW];
  bwd_pair<T, BM, BN, 2>(gd, ed, gw, ew, nw, smem);
}

int xcd_group(int gm, int gn, int split, int bm, int bn) {
  // one XCD's range: L tiles from the start of a split-K slice
  const int64_t per = int64_t(gm) * gn;
  const int64_t L = std::max<int64_t>(1, std::min<int64_t>(per, per * split / kXcds));
  int best = 1;
  int64_t bestc = INT64_MAX;
  for (int g = 1; g <= gm; ++g) {
    int64_t mc, nc;
    if (L <= int64_t(g) * gn) {
      mc = std::min<int64_t>(g, L);
      nc = (L + g - 1) / g;
    } else {
      mc = std::min<int64_t>(gm, (L + int64_t(g) * gn - 1) / (int64_t(g) * gn) * g);
      nc = gn;
    }
    const int64_t c = mc * bm + nc * bn;
    if (c < bestc) {
      bestc = c;
      best = g;
    }
  }
  return best;
}

static GemmDesc with_group(const GemmDesc& g0, int BM, int BN) {
  GemmDesc g = g0;
  if (g.group <= 0) g.group = xcd_group((g.M + BM - 1) / BM, (g.N + BN - 1) / BN, g.split, BM, BN);
  return g;
}

// bf16 first-layer weight gradient with its Adam update (eight waves per
// tile) and the Adam chunks of `a` (none when a.nchunks is 0)
static hipError_t launch_wgrad_w8(const GemmDesc& g, const EpiParams& e, const AdamArgs& a, hipStream_t s,
                                  const LaunchEv& ev);

template <typename T, int BM, int BN>
static hipError_t launch_gemm_t(int kind, const GemmDesc& g0, const EpiParams& e, hipStream_t s, const LaunchEv& ev) {
  const GemmDesc g = with_group(g0, BM, BN);
  dim3 grid(((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN) * g.split), block(256);
  // the fused Adam update exists only in the two k-group weight gradient
  if (kind == GK_WGRAD && e.ap && (g.kgroups != 2 || g.split != 1)) return hipErrorInvalidValue;
  if (g.kgroups == 2) {
    // two k-groups: the unsplit 64x64 weight gradient (fp32 or bf16)
    if constexpr (BM == 64 && BN == 64) {
      if (kind == GK_WGRAD && g.split == 1) {
        // bf16: the eight-wave tiles of the launch that also updates the
        // block's other parameters (the same sums, so every schedule gives
        // the same bits), here without those; they need the fused update
        if constexpr (sizeof(T) == 2) return e.ap ? launch_wgrad_w8(g, e, AdamArgs{}, s, ev) : hipErrorInvalidValue;
        ERASE_LAUNCH((erase_wgrad_gemm_kg2<T, BM, BN>), grid, dim3(512), 0, s, ev, g, e);
        return hipGetLastError();
      }
    }
    // and bf16 64x128 and 64x64 forward tiles
    if constexpr (sizeof(T) == 2 && BM == 64 && (BN == 128 || BN == 64)) {
      if (kind == GK_FWD_RELU) {
        ERASE_LAUNCH((erase_fwd_gemm_kg2<T, BM, BN>), grid, dim3(512), 0, s, ev, g, e);
        return hipGetLastError();
      }
      if (kind == GK_FWD_CROSS) {
        ERASE_LAUNCH((erase_fwd_cross_gemm_kg2<T, BM, BN>), grid, dim3(512), 0, s, ev, g, e);
        return hipGetLastError();
      }
    }
    return hipErrorInvalidValue;
  }
  switch (kind) {
    case GK_FWD_RELU: ERASE_LAUNCH((erase_fwd_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e); break;
    case GK_FWD_CROSS: ERASE_LAUNCH((erase_fwd_cross_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e); break;
    case GK_WGRAD:
      if constexpr (BM >= 64) {  // k-major tiles of 64 or 128 columns
        ERASE_LAUNCH((erase_wgrad_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e);
      } else {
        return hipErrorInvalidValue;
      }
      break;
    case GK_DGRAD: ERASE_LAUNCH((erase_dgrad_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e); break;
    case GK_FWD_LIN:
    case GK_FWD_GELU:
    case GK_DGRAD_GELU:
    case GK_FWD_LOGITS:
      // transformer kinds: bf16, 64- and 128-row tiles
      if constexpr (sizeof(T) == 2 && BM >= 64) {
        if (kind == GK_FWD_LIN) ERASE_LAUNCH((erase_fwd_lin_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e);
        if (kind == GK_FWD_GELU) ERASE_LAUNCH((erase_fwd_gelu_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e);
        if (kind == GK_DGRAD_GELU) ERASE_LAUNCH((erase_dgrad_gelu_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e);
        if (kind == GK_FWD_LOGITS) ERASE_LAUNCH((erase_fwd_logits_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e);
      } else {
        return hipErrorInvalidValue;
      }
      break;
    case GK_FWD_HEAD:
      // the tile must span the whole width; 32- and 64-row tiles only
      if constexpr (BM <= 64) {
        if (g.N > BN) return hipErrorInvalidValue;
        ERASE_LAUNCH((erase_fwd_head_gemm<T, BM, BN>), grid, block, 0, s, ev, g, e);
      } else {
        return hipErrorInvalidValue;
      }
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int BM, int BN, int KG = 1>
static hipError_t launch_bwd_t(const GemmDesc& gd0, const EpiParams& ed, const GemmDesc& gw0, const EpiParams& ew,
                               hipStream_t s, const LaunchEv& ev) {
  const GemmDesc gd = with_group(gd0, BM, BN), gw = with_group(gw0, BM, BN);
  const int nd = ((gd.M + BM - 1) / BM) * ((gd.N + BN - 1) / BN);
  const int nw = ((gw.M + BM - 1) / BM) * ((gw.N + BN - 1) / BN) * gw.split;
  // 128x128: one workgroup per CU (an unused dynamic LDS reservation): two
  // co-resident 128x128 workgroups measured 20% slower on the vocabulary
  // head's backward (1.69 vs 1.41 ms)
  if constexpr (KG == 2) {
    ERASE_LAUNCH((erase_bwd_gemm_kg2<T, BM, BN>), dim3(nd + nw), dim3(512), 0, s, ev, gd, ed, gw, ew, nw);
    return hipGetLastError();
  }
  constexpr size_t kReserve = BM == 128 ? 40960 : 0;
  if constexpr (kReserve > 0) {
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&erase_bwd_gemm<T, BM, BN>), hipFuncAttributeMaxDynamicSharedMemorySize,
        (int)kReserve);
    if (attr != hipSuccess) return attr;
  }
  ERASE_LAUNCH((erase_bwd_gemm<T, BM, BN>), dim3(nd + nw), dim3(256), kReserve, s, ev, gd, ed, gw, ew, nw);
  return hipGetLastError();
}

hipError_t launch_bwd_gemm(int bf16, const GemmDesc& gd, const EpiParams& ed, const GemmDesc& gw, const EpiParams& ew,
                           hipStream_t s, const LaunchEv& ev) {
  if (gd.bm != gw.bm || gd.bn != gw.bn || gd.split != 1 || gw.split <= 0 || ew.ap) return hipErrorInvalidValue;
  if (gd.kgroups == 2 || gw.kgroups == 2) {  // two k-groups: bf16 128x128 only
    if (!bf16 || gd.kgroups != gw.kgroups || gd.bm != 128 || gd.bn != 128) return hipErrorInvalidValue;
    return launch_bwd_t<uint16_t, 128, 128, 2>(gd, ed, gw, ew, s, ev);
  }
  if (bf16) {
    if (gd.bm == 128 && gd.bn == 128) return launch_bwd_t<uint16_t, 128, 128>(gd, ed, gw, ew, s, ev);
    if (gd.bm == 64 && gd.bn == 64) return launch_bwd_t<uint16_t, 64, 64>(gd, ed, gw, ew, s, ev);
  } else {
    if (gd.bm == 64 && gd.bn == 64) return launch_bwd_t<float, 64, 64>(gd, ed, gw, ew, s, ev);
  }
  return hipErrorInvalidValue;
}

// The last layer of a block with its local head and loss (Section 2.1,
// Eq. 2) for bf16 outputs at most 128 wide, in 16-row tiles: twice as many
// workgroups as the 32-row GEMM-core tile, for a layer whose work is a few
// k-steps.  Four waves of 32 output columns each; the MFMA operands come
// straight from global memory (the rows of the activation and of the weight
// copy are contiguous along the contraction, and every load of the
// contraction is in flight at once, up to 256 per pass).  Per tile:
//   z = relu(acc + b) (as stored, bf16),  s_m = sum_n z_mn w_n + c,
//   loss_m = max(s,0) - s y_m + log1p(e^-|s|),  ds_m = lam (sigmoid(s_m) - y_m) / M,
//   dz_mn = ds_m w_n [z_mn > 0],  partials dw_n = sum_m z_mn ds_m, dc, loss,
// every sum in a fixed order.
__global__ __launch_bounds__(256) void erase_fwd_head16(GemmDesc g, EpiParams e) {
  constexpr int TR = 16, TC = 128, OP = TC + 8;  // tile rows, columns, LDS pitch (bf16)
  __shared__ float s_part[4][TR];
  __shared__ float s_ds[TR], s_l[TR];
  __shared__ __attribute__((aligned(16))) uint16_t s_z[TR][OP];
  __shared__ __attribute__((aligned(16))) uint16_t s_dz[TR][OP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = g.M, N = g.N, K = g.K;
  const int m0 = (int)blockIdx.x * TR;
  const int fr = lane & 15, kq = (lane >> 4) * 8;
  const int c0 = wave * 32 + fr, c1 = c0 + 16;  // this lane's two output columns
  const uint16_t* A = static_cast<const uint16_t*>(g.A);
  const uint16_t* W = static_cast<const uint16_t*>(g.B);
  const uint16_t* pa = A + (int64_t)(m0 + fr) * g.lda + kq;
  const uint16_t* pb0 = W + (int64_t)c0 * g.ldb + kq;
  const uint16_t* pb1 = W + (int64_t)c1 * g.ldb + kq;
  // head inputs first: their latency hides behind the operand loads
  const float b0 = c0 < N ? e.bias[c0] : 0.f, b1 = c1 < N ? e.bias[c1] : 0.f;
  const float w0 = c0 < N ? e.hw[c0] : 0.f, w1 = c1 < N ? e.hw[c1] : 0.f;
  const float hc = e.hc[0];
  float yl = 0.f;
  if (tid < TR && m0 + tid < M) yl = e.labels[m0 + tid];
  f32x4_t acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < K; k0 += 8 * 32) {
    u32x4_t fa[8], f0[8], f1[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (k0 + 32 * u < K) {
        fa[u] = *reinterpret_cast<const u32x4_t*>(pa + k0 + 32 * u);
        f0[u] = *reinterpret_cast<const u32x4_t*>(pb0 + k0 + 32 * u);
        f1[u] = *reinterpret_cast<const u32x4_t*>(pb1 + k0 + 32 * u);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (k0 + 32 * u < K) {
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[u]),
                                                       __builtin_bit_cast(bf16x8_t, f0[u]), acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[u]),
                                                       __builtin_bit_cast(bf16x8_t, f1[u]), acc1, 0, 0, 0);
      }
    }
  }
  // lane holds rows 4 (lane >> 4) + q of columns c0 and c1
  const int rb = (lane >> 4) * 4;
  float z0[4], z1[4], part[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool live = m0 + rb + q < M;
    const float v0 = acc0[q] + b0, v1 = acc1[q] + b1;
    z0[q] = (live && c0 < N) ? bf2f(f2bf(v0 < 0.f ? 0.f : v0)) : 0.f;  // keeps NaN, like max(h, 0)
    z1[q] = (live && c1 < N) ? bf2f(f2bf(v1 < 0.f ? 0.f : v1)) : 0.f;
    part[q] = fmaf(z1[q], w1, z0[q] * w0);
  }
  // the row's partial logit over the wave's 32 columns: lanes of one row
  // group (16 lanes) combined by a fixed butterfly
#pragma unroll
  for (int q = 0; q < 4; ++q) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) part[q] += __shfl_xor(part[q], o, 64);
    if (fr == 0) s_part[wave][rb + q] = part[q];
  }
  __syncthreads();
  if (tid < TR) {
    float ds = 0.f, l = 0.f;
    if (m0 + tid < M) {
      const float sv = ((s_part[0][tid] + s_part[1][tid]) + (s_part[2][tid] + s_part[3][tid])) + hc;
      const float en = __expf(-fabsf(sv));
      const float sig = sv >= 0.f ? 1.f / (1.f + en) : en / (1.f + en);
      ds = e.lam * (sig - yl) * e.inv_m;
      l = fmaxf(sv, 0.f) - sv * yl + log1pf(en);
    }
    s_ds[tid] = ds;
    s_l[tid] = l;
  }
  __syncthreads();
  float dw0 = 0.f, dw1 = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float ds = s_ds[rb + q];
    s_z[rb + q][c0] = f2bf(z0[q]);
    s_z[rb + q][c1] = f2bf(z1[q]);
    s_dz[rb + q][c0] = f2bf(z0[q] > 0.f ? ds * w0 : 0.f);
    s_dz[rb + q][c1] = f2bf(z1[q] > 0.f ? ds * w1 : 0.f);
    dw0 = fmaf(z0[q], ds, dw0);
    dw1 = fmaf(z1[q], ds, dw1);
  }
  // column sums over the tile's 16 rows: the four row groups (lanes 16 apart)
  dw0 += __shfl_xor(dw0, 16, 64);
  dw0 += __shfl_xor(dw0, 32, 64);
  dw1 += __shfl_xor(dw1, 16, 64);
  dw1 += __shfl_xor(dw1, 32, 64);
  if (lane < 16) {
    if (c0 < N) e.pdw[(int64_t)blockIdx.x * N + c0] = dw0;
    if (c1 < N) e.pdw[(int64_t)blockIdx.x * N + c1] = dw1;
  }
  if (tid == 0) {
    float d = 0.f, l = 0.f;
    for (int r = 0; r < TR; ++r) {
      d += s_ds[r];
      l += s_l[r];
    }
    e.pdc[blockIdx.x] = d;
    e.ploss[blockIdx.x] = l;
  }
  __syncthreads();
  // 16-byte row-major stores of dz (and of z when a later block reads it)
  const int r = tid >> 4, n = (tid & 15) * 8;
  if (m0 + r < M && n < N) {
    if (e.dmn) {
      uint16_t* dst = static_cast<uint16_t*>(e.dmn) + (int64_t)(m0 + r) * e.lddmn + n;
      if (n + 8 <= N)
        *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(&s_dz[r][n]);
      else
        for (int k = 0; k < N - n; ++k) dst[k] = s_dz[r][n + k];
    }
    if (e.y) {
      uint16_t* dst = static_cast<uint16_t*>(e.y) + (int64_t)(m0 + r) * e.ldy + n;
      if (n + 8 <= N)
        *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(&s_z[r][n]);
      else
        for (int k = 0; k < N - n; ++k) dst[k] = s_z[r][n + k];
    }
  }
}

// bf16 vocabulary logits in 256x256 tiles; false when the shape does not fit
static bool logits_wide_fits(const GemmDesc& g, const EpiParams& e);
static hipError_t launch_logits_wide(const GemmDesc& g, const EpiParams& e, hipStream_t s, const LaunchEv& ev);

hipError_t launch_gemm(int bf16, int kind, const GemmDesc& g, const EpiParams& e, hipStream_t s, const LaunchEv& ev) {
  if (g.M <= 0 || g.N <= 0 || g.split <= 0) return hipErrorInvalidValue;
  if (bf16 && kind == GK_FWD_LOGITS && g.bm == 256 && g.bn == 256)
    return logits_wide_fits(g, e) ? launch_logits_wide(g, e, s, ev) : hipErrorInvalidValue;
  if (bf16 && kind == GK_FWD_HEAD && g.bm == 16) {
    // 16-row tiles: outputs at most 128 wide, contraction a multiple of 32
    if (g.N > 128 || g.K % 32 || g.split != 1) return hipErrorInvalidValue;
    ERASE_LAUNCH(erase_fwd_head16, dim3((unsigned)((g.M + 15) / 16)), dim3(256), 0, s, ev, g, e);
    return hipGetLastError();
  }
  if (bf16) {
    if (g.bm == 128 && g.bn == 128) return launch_gemm_t<uint16_t, 128, 128>(kind, g, e, s, ev);
    if (g.bm == 128 && g.bn == 64) return launch_gemm_t<uint16_t, 128, 64>(kind, g, e, s, ev);
    if (g.bm == 64 && g.bn == 128) return launch_gemm_t<uint16_t, 64, 128>(kind, g, e, s, ev);
    if (g.bm == 64 && g.bn == 64) return launch_gemm_t<uint16_t, 64, 64>(kind, g, e, s, ev);
    if (g.bm == 32 && g.bn == 128 && kind == GK_FWD_HEAD) return launch_gemm_t<uint16_t, 32, 128>(kind, g, e, s, ev);
  } else {
    if (g.bm == 64 && g.bn == 64) return launch_gemm_t<float, 64, 64>(kind, g, e, s, ev);
  }
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// step prologue: t += 1, xp = x (zero-padded copy) and xt = x^T, through a
// 64 x 64 LDS tile with 16-byte global loads and stores
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void erase_prologue(PrologueArgs a) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const int64_t t = a.t[0] + 1;
    a.t[0] = t;
    a.hyper[0] = (float)((double)a.lr / (1.0 - pow((double)a.beta1, (double)t)));
    a.hyper[1] = (float)sqrt(1.0 - pow((double)a.beta2, (double)t));
  }
  if (a.xp == nullptr) return;
  // xp[m][k] = x[m][k] for k < K, zero for the rest of the 16-byte chunk;
  // columns past the chunk and rows past M stay zero from initialisation
  constexpr int KCH = 16 / sizeof(T);
  const T* X = static_cast<const T*>(a.x);
  const int cpr = (a.K + KCH - 1) / KCH;  // chunks per row
  const int64_t nch = (int64_t)a.M * cpr;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < nch; c += (int64_t)gridDim.x * 256) {
    const int m = (int)(c / cpr), k = (int)(c - (int64_t)m * cpr) * KCH;
    // x rows hold at least roundup(K, KCH) elements (16-byte row pitch)
    uint4 v = *reinterpret_cast<const uint4*>(X + (int64_t)m * a.ldx + k);
    if (k + KCH > a.K) {
      T e[KCH];
      __builtin_memcpy(e, &v, 16);
#pragma unroll
      for (int q = 0; q < KCH; ++q)
        if (k + q >= a.K) e[q] = T(0);
      __builtin_memcpy(&v, e, 16);
    }
    *reinterpret_cast<uint4*>(static_cast<T*>(a.xp) + (int64_t)m * a.ldxp + k) = v;
  }
}

hipError_t launch_prologue(int bf16, const PrologueArgs& a, hipStream_t s, const LaunchEv& ev) {
  const int64_t nch = a.xp ? (int64_t)a.M * ((a.K + 16 / (bf16 ? 2 : 4) - 1) / (16 / (bf16 ? 2 : 4))) : 1;
  dim3 grid((unsigned)std::min<int64_t>((nch + 255) / 256, 4096)), block(256);
  if (bf16)
    ERASE_LAUNCH(erase_prologue<uint16_t>, grid, block, 0, s, ev, a);
  else
    ERASE_LAUNCH(erase_prologue<float>, grid, block, 0, s, ev, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// local head + sigmoid-BCE + gradient at z.  One workgroup stages R rows of z
// ([R][N] tile in LDS, 16-byte global loads), then:
//   s_i = z_i . w + c, l_i = max(s,0) - s y + log1p(e^-|s|),
//   ds_i = lam (sigmoid(s_i) - y_i) / M,
//   dz = ds_i w_n [z_in > 0]  (row-major and feature-major, 16-byte stores),
//   partial dw_n = sum_i z_in ds_i, partial dc = sum_i ds_i, partial loss,
// every sum in a fixed order.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void erase_head_bce(HeadArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  constexpr int KCH = 16 / sizeof(T);  // elements per 16-byte chunk
  __shared__ float s_ds[32];
  __shared__ float s_loss[32];
  __shared__ float s_w[HEAD_MAX_N];
  T* tile = reinterpret_cast<T*>(smem_raw);
  const int N = a.N;
  const int R = head_rows(N, sizeof(T));
  const int pitch = head_pitch(N, sizeof(T));
  const int tid = threadIdx.x;
  const int r0 = blockIdx.x * R;
  const int rows = min(R, a.M - r0);
  const T* Z = static_cast<const T*>(a.z);
  const int cpr = (N + KCH - 1) / KCH;  // chunks per row

  for (int n = tid; n < N; n += 256) s_w[n] = a.w[n];
  // stage the tile (rows beyond M and columns beyond N are zero)
  for (int c = tid; c < R * cpr; c += 256) {
    const int r = c / cpr, k = (c - r * cpr) * KCH;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (r < rows) {
      const T* p = Z + (int64_t)(r0 + r) * a.ldz + k;
      if (k + KCH <= N) {
        v = *reinterpret_cast<const uint4*>(p);
      } else {
        T tmp[KCH];
#pragma unroll
        for (int e = 0; e < KCH; ++e) tmp[e] = (k + e < N) ? p[e] : T(0);
        __builtin_memcpy(&v, tmp, 16);
      }
    }
    *reinterpret_cast<uint4*>(&tile[r * pitch + k]) = v;
  }
  __syncthreads();

  // logits: 256/R lanes per row, then a fixed butterfly over those lanes
  {
    const int tpr = 256 / R;  // power of two, 8..64
    const int r = tid / tpr, j = tid - r * tpr;
    float part = 0.f;
    for (int n = j; n < N; n += tpr) part = fmaf(asf(tile[r * pitch + n]), s_w[n], part);
    for (int off = 1; off < tpr; off <<= 1) part += __shfl_xor(part, off, 64);
    if (j == 0) {
      float ds = 0.f, l = 0.f;
      if (r < rows) {
        const float s = part + a.c[0];
        const float yv = a.y[r0 + r];
        const float en = __expf(-fabsf(s));
        const float sig = s >= 0.f ? 1.f / (1.f + en) : en / (1.f + en);
        ds = a.lam * (sig - yv) * a.inv_m;
        l = fmaxf(s, 0.f) - s * yv + log1pf(en);
      }
      s_ds[r] = ds;
      s_loss[r] = l;
    }
  }
  __syncthreads();

  // dz row-major
  if (a.dmn) {
    T* D = static_cast<T*>(a.dmn);
    for (int c = tid; c < rows * cpr; c += 256) {
      const int r = c / cpr, k = (c - r * cpr) * KCH;
      const float ds = s_ds[r];
      T o[KCH];
#pragma unroll
      for (int e = 0; e < KCH; ++e) {
        const float zv = asf(tile[r * pitch + k + e]);
        o[e] = cvt<T>((zv > 0.f && k + e < N) ? ds * s_w[min(k + e, N - 1)] : 0.f);
      }
      T* p = D + (int64_t)(r0 + r) * a.lddmn + k;
      if (k + KCH <= N) {
        uint4 v;
        __builtin_memcpy(&v, o, 16);
        *reinterpret_cast<uint4*>(p) = v;
      } else {
        for (int e = 0; e < KCH && k + e < N; ++e) p[e] = o[e];
      }
    }
  }
  // partial head gradients and loss of this workgroup's rows
  for (int n = tid; n < N; n += 256) {
    float acc = 0.f;
    for (int r = 0; r < rows; ++r) acc = fmaf(asf(tile[r * pitch + n]), s_ds[r], acc);
    a.pdw[(int64_t)blockIdx.x * N + n] = acc;
  }
  if (tid == 0) {
    float sd = 0.f, sl = 0.f;
    for (int r = 0; r < rows; ++r) {
      sd += s_ds[r];
      sl += s_loss[r];
    }
    a.pdc[blockIdx.x] = sd;
    a.ploss[blockIdx.x] = sl;
  }
}

hipError_t launch_head(int bf16, const HeadArgs& a, hipStream_t s, const LaunchEv& ev) {
  const int esz = bf16 ? 2 : 4;
  dim3 grid((a.M + head_rows(a.N, esz) - 1) / head_rows(a.N, esz)), block(256);
  const size_t lds = head_lds_bytes(a.N, esz);
  if (bf16)
    ERASE_LAUNCH(erase_head_bce<uint16_t>, grid, block, (uint32_t)lds, s, ev, a);
  else
    ERASE_LAUNCH(erase_head_bce<float>, grid, block, (uint32_t)lds, s, ev, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Adam over all parameter segments of one block (one ADAM_TR x ADAM_TC tile
// per workgroup), with the ordered reduction of split partials fused in
// front and the GEMM copies of the updated weights written behind.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_seg(const AdamArgs& a, int64_t chunk) {
  int s = 0;
  while (s + 1 < a.nseg && a.chunk0[s + 1] <= chunk) ++s;
  return s;
}

// A matrix tile is ADAM_TR rows of ADAM_TC columns: rows are read and
// written coalesced across the workgroup, and the transposed GEMM copy gets
// the tile's ADAM_TR consecutive values of each column from one thread
// (32 contiguous bytes in bf16).
// 16-byte access at 4-byte alignment (rows of the flat parameter arrays
// start anywhere; gfx950 serves unaligned vector accesses)
typedef float f32x4u_t __attribute__((ext_vector_type(4), aligned(4)));


// One chunk of the Adam launch (ADAM_TR x ADAM_TC of a matrix segment, or
// ADAM_TC elements of a vector) by 256 threads (tid 0..255) of a workgroup,
// and the block loss with chunk 0.  s_o stages this chunk's transposed copy.
// Every call executes exactly one __syncthreads (whatever the segment kind;
// a negative chunk only takes part in it), so the two halves of a
// 512-thread workgroup can each run a chunk.
template <typename T>
__device__ __forceinline__ void adam_chunk(const AdamArgs& a, int64_t chunk, int tid, T (*s_o)[ADAM_TC]) {
  if (chunk < 0) {
    __syncthreads();
    return;
  }
  const AdamSeg sg = a.seg[find_seg(a, chunk)];
  bool trans = false;  // the transposed copy is stored after the barrier
  int r0 = 0, tile = 0;
  const float step = a.hyper[0];  // lr / (1 - beta1^t)
  const float bc2s = a.hyper[1];  // sqrt(1 - beta2^t)
  const float b1 = a.beta1, b2 = a.beta2, eps = a.eps;
  tile = (int)(chunk - sg.chunk0);
  auto P = gmem(sg.p);
  auto Mo = gmem(sg.m);
  auto V = gmem(sg.v);
  auto PART = gmem(sg.part);

  if (sg.rows == 1) {
    // a vector (bias or head parameter): one element per thread, possibly
    // many partials (one per head workgroup), 32 loads in flight per batch,
    // added in slice order
    const int c = tile * ADAM_TC + tid;
    const bool ok = tid < ADAM_TC && c < sg.cols;
    const int cc = ok ? c : 0;  // clamped: loads stay in bounds
    float p = P[cc], m = Mo[cc], v = V[cc], g = 0.f;
    constexpr int ZV = 32;
    for (int z0 = 0; z0 < sg.nsplit; z0 += ZV) {
      float tv[ZV];
#pragma unroll
      for (int j = 0; j < ZV; ++j) tv[j] = (z0 + j < sg.nsplit) ? PART[cc + (int64_t)(z0 + j) * sg.pstride] : 0.f;
#pragma unroll
      for (int j = 0; j < ZV; ++j)
        if (z0 + j < sg.nsplit) g += tv[j];
    }
    adam_elem(p, m, v, g, b1, b2, step, bc2s, eps);
    if (ok) {
      if (sg.g) gmem(sg.g)[c] = g;
      Mo[c] = m;
      V[c] = v;
      P[c] = p;
      if (sg.sh) gmem(static_cast<T*>(sg.sh))[c] = cvt<T>(p);
    }
  } else {
    // a matrix: a workgroup covers ADAM_TR (16) rows x ADAM_TC (64) columns,
    // a thread 4 consecutive columns of one row (16-byte loads and stores)
    static_assert(ADAM_TR == 16 && ADAM_TC == 64, "matrix tile is 16 rows x 16 threads x 4 columns");
    r0 = (tile / sg.tcols) * ADAM_TR;
    const int r = r0 + (tid >> 4);
    const int c0 = (tile % sg.tcols) * ADAM_TC + (tid & 15) * 4;
    const bool any = r < sg.rows && c0 < sg.cols;
    const bool full = c0 + 4 <= sg.cols;
    const int rr = any ? r : 0, cc = any ? c0 : 0;  // clamped: loads stay in bounds
    const int64_t fi = (int64_t)rr * sg.cols + cc;
    // split partials: rows padded to a multiple of 64 columns, so the 4
    // columns from c0 are in bounds and 16-byte aligned
    const int64_t po = (int64_t)rr * sg.ldpart + cc;
    // Ordered reduction of the split partials, slices added in order 0, 1,
    // ...  Four slices per batch; the first batch is issued together with the
    // parameter loads.  Slices past the last one are clamped loads added as
    // zeros (a select, not a branch, so no wait splits a batch).
    constexpr int ZS = 4;
    f32x4_t tv[ZS];
    auto load_batch = [&](int z0) {
#pragma unroll
      for (int j = 0; j < ZS; ++j)
        tv[j] = *reinterpret_cast<const __attribute__((address_space(1))) f32x4_t*>(
            PART + (int64_t)min(z0 + j, sg.nsplit - 1) * sg.pstride + po);
    };
    float g[4] = {0.f, 0.f, 0.f, 0.f};
    auto add_batch = [&](int z0) {
#pragma unroll
      for (int j = 0; j < ZS; ++j) {
        const bool in = z0 + j < sg.nsplit;
#pragma unroll
        for (int k = 0; k < 4; ++k) g[k] += in ? tv[j][k] : 0.f;
      }
    };
    load_batch(0);
    // Unconditional 16-byte loads (no branch, so they are all in flight
    // together).  At a row's ragged end they read up to 3 elements past the
    // row; past the matrix's last row that is its bias and the head, which
    // follow every weight matrix in the block's flat arrays (at least 3
    // elements), so the loads stay in bounds.  Only stores are masked.
    const f32x4u_t pv = *reinterpret_cast<const __attribute__((address_space(1))) f32x4u_t*>(P + fi);
    const f32x4u_t mv = *reinterpret_cast<const __attribute__((address_space(1))) f32x4u_t*>(Mo + fi);
    const f32x4u_t vv = *reinterpret_cast<const __attribute__((address_space(1))) f32x4u_t*>(V + fi);
    add_batch(0);
    for (int z0 = ZS; z0 < sg.nsplit; z0 += ZS) {
      load_batch(z0);
      add_batch(z0);
    }
    float p[4], m[4], v[4];
    T o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      p[k] = pv[k];
      m[k] = mv[k];
      v[k] = vv[k];
      adam_elem(p[k], m[k], v[k], g[k], b1, b2, step, bc2s, eps);
      o[k] = cvt<T>(p[k]);
    }
    if (any) {
      if (full) {
        auto st = [&](float* base, const float* x) {
          f32x4u_t w = {x[0], x[1], x[2], x[3]};
          __builtin_nontemporal_store(w, reinterpret_cast<__attribute__((address_space(1))) f32x4u_t*>(gmem(base) + fi));
        };
        if (sg.g) st(sg.g, g);
        st(sg.m, m);
        st(sg.v, v);
        st(sg.p, p);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (c0 + k < sg.cols) {
            if (sg.g) gmem(sg.g)[fi + k] = g[k];
            Mo[fi + k] = m[k];
            V[fi + k] = v[k];
            P[fi + k] = p[k];
          }
      }
      // GEMM copy [rows][ldsh]: 4 columns of row r
      if (sg.sh) {
        T* D = static_cast<T*>(sg.sh) + (int64_t)r * sg.ldsh + c0;
        if (full) {
          st4(D, o);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (c0 + k < sg.cols) D[k] = o[k];
        }
      }
    }
    // transposed GEMM copy [cols][ldsht]: the 16 rows of each column, through
    // LDS (one thread per column, four 4-element stores)
    if (sg.sht) {
      const int cl = (tid & 15) * 4, rl = tid >> 4;
#pragma unroll
      for (int k = 0; k < 4; ++k) s_o[rl][cl + k] = o[k];
      trans = true;
    }
  }
  __syncthreads();
  if (trans && tid < ADAM_TC) {
    const int c = (tile % sg.tcols) * ADAM_TC + tid;
    if (c < sg.cols && r0 < sg.rows) {
      T* D = static_cast<T*>(sg.sht) + (int64_t)c * sg.ldsht + r0;
#pragma unroll
      for (int q4 = 0; q4 < ADAM_TR; q4 += 4) {
        T t4[4] = {s_o[q4][tid], s_o[q4 + 1][tid], s_o[q4 + 2][tid], s_o[q4 + 3][tid]};
        if (r0 + q4 + 4 <= sg.rows) {
          st4(D + q4, t4);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (r0 + q4 + i < sg.rows) D[q4 + i] = t4[i];
        }
      }
    }
  }
  if (chunk == 0 && tid < 64 && a.ploss) {
    // block loss: lane l sums partials l, l+64, ... in order, then a fixed
    // butterfly across the wave
    float L = 0.f;
    for (int i = tid; i < a.nloss; i += 64) L += a.ploss[i];
    L = wave_sum(L) * a.inv_m;
    if (tid == 0) {
      a.loss_out[0] = L;
      if (!(fabsf(L) <= 3.4e38f)) a.status[0] = 1;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void erase_adam(AdamArgs a) {
  __shared__ T s_o[ADAM_TR][ADAM_TC];
  adam_chunk<T>(a, blockIdx.x, (int)threadIdx.x, s_o);
}

// A block's first-layer weight gradient with its fused Adam (two k-groups,
// unsplit) and, in the same launch, the Adam update of the block's other
// parameters: workgroups [0, ntiles) are the GEMM tiles (one per CU at
// most), the rest run two Adam chunks each (one per half of the workgroup)
// on the CUs the tiles leave free.  The two parts touch disjoint parameters,
// and the Adam part reads only gradients finished by earlier launches.
template <typename T, int BM, int BN>
__global__ __launch_bounds__(512) void erase_wgrad_adam_kg2(GemmDesc g, EpiParams e, AdamArgs a, int ntiles) {
  constexpr int BKK = sizeof(T) == 2 ? 128 : 0;
  __shared__ __attribute__((aligned(16))) char smem[GemmSmem<T, BM, BN, GK_WGRAD, BKK>::BYTES];
  static_assert(GemmSmem<T, BM, BN, GK_WGRAD, BKK>::BYTES >= 2 * ADAM_TR * ADAM_TC * (int)sizeof(T), "staging");
  const int b = blockIdx.x;
  if (b < ntiles) {
    const int gm = (g.M + BM - 1) / BM, gn = (g.N + BN - 1) / BN;
    const TileIdx ti = tile_from(xcd_linear(b, ntiles), gm, gn, g.group);
    gemm_body<T, BM, BN, GK_WGRAD, 2, 2, BKK>(g, e, ti.m, ti.n, ti.z, smem);
  } else {
    const int half = (int)threadIdx.x >> 8;
    T(*s_o)[ADAM_TC] = reinterpret_cast<T(*)[ADAM_TC]>(smem) + half * ADAM_TR;
    const int64_t chunk = 2 * (int64_t)(b - ntiles) + half;
    adam_chunk<T>(a, chunk < a.nchunks ? chunk : -1, (int)threadIdx.x & 255, s_o);
  }
}

// ---------------------------------------------------------------------------
// The same launch for bf16: four waves per 64x64 tile, no barrier in the main
// loop, operands loaded straight into LDS.  Every wave owns the whole tile
// and contracts its own 32 rows of each 128-row k-step (one MFMA k-step over
// 16 independent 16x16 accumulators).  It loads exactly those rows of both
// operands into two LDS slices of its own with global_load_lds_dwordx4 (no
// registers hold data in flight, no LDS store instructions) and reads its
// fragments back with the transposing read, so no wave waits for another
// until the partial tiles are added.  The loads of k-step j + 1 are in
// flight while k-step j is read and multiplied.  Measured at 512 x 1677 over
// 4096 rows (GEMM part): 15.1 us, against 23 us for two k-groups of four waves
// with a barrier per k-step and 15.5 us for eight waves staging through
// registers.
// The four partial tiles are added through LDS in wave order, and the
// finished tile goes through the Adam update as above.
namespace w4 {
constexpr int BM = 64, BN = 64;        // output tile: dW rows (dH features) x columns (X features)
constexpr int NW = 4, NT = 64 * NW;    // waves and threads per workgroup
constexpr int KW = 32;                 // batch rows per wave and k-step: one MFMA k-step
constexpr int BK = KW * NW;            // batch rows per k-step
constexpr int SLICE = KW * (BM + BN);  // bf16 elements of one LDS slice of a wave (8 KB)
constexpr int RED = NW * BM * BN;      // the waves' fp32 partial tiles (64 KB)
constexpr int MAIN = NW * 2 * SLICE * 2 > RED * 4 ? NW * 2 * SLICE * 2 : RED * 4;
constexpr int BYTES = MAIN + NW * BM * 4;  // and each wave's bias row sums
constexpr int IT = BM * BN / (4 * NT);     // Adam items of 4 columns per thread
}  // namespace w4

// k-major rows r of 8 chunks are stored with chunk j at j ^ kperm8(r) (the
// permutation of the GEMM core's k-major tiles)
__device__ __forceinline__ int kperm8(int r) { return 2 * ((r >> 1) & 1) + 4 * ((r >> 3) & 1); }

// One 16-byte chunk per lane from global memory straight into LDS: lane l
// writes bytes [lds + 16 l, lds + 16 l + 16) of the wave's 1 KB block at the
// LDS byte address `lds` (wave-uniform, through M0).  The load counts in the
// wave's vector-memory counter like any load; the caller waits for it before
// reading the block.  The compiler reserves M0 and keeps nothing in it across
// these statements: no other instruction of the kernel reads it.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src) : "memory");
}
// The same with a wave-uniform base address in scalar registers and the
// lane's 32-bit byte offset from it (no 64-bit address per lane and load).
__device__ __forceinline__ void lds_dma16s(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(off), "s"(base) : "memory");
}

__device__ __forceinline__ void wgrad_adam_w4_tile(const GemmDesc& g, const EpiParams& e, int bx, int by,
                                                   char* smem) {
  using namespace w4;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m0 = bx * BM, n0 = by * BN;
  const int K = g.K;  // a multiple of 64: a wave's 32-row slice is wholly in or past it
  const uint16_t* A = static_cast<const uint16_t*>(g.A);
  const uint16_t* B = static_cast<const uint16_t*>(g.B);

  const bool do_rows = e.bpart != nullptr && by == 0;
  float rs[4] = {0.f, 0.f, 0.f, 0.f};
  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // The wave's slices: A rows (dH, 32 x 64) then B rows (X, 32 x 64), rows
  // of 128 bytes.  Load u of an operand fills slice rows 8u..8u+7: lane l
  // writes row 8u + (l >> 3), chunk slot l & 7, which holds the row's chunk
  // (l & 7) ^ kperm8(row).
  const int lr = lane >> 3, lc = lane & 7;
  const uint16_t* pa[4];
  const uint16_t* pb[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int r = 8 * u + lr, ch = lc ^ kperm8(r);
    pa[u] = A + (int64_t)(KW * wv + r) * g.lda + m0 + ch * 8;
    pb[u] = B + (int64_t)(KW * wv + r) * g.ldb + n0 + ch * 8;
  }
  const int64_t ka = (int64_t)BK * g.lda, kb = (int64_t)BK * g.ldb;
  uint16_t* mine = reinterpret_cast<uint16_t*>(smem) + wv * 2 * SLICE;
  const uint32_t lmine = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) uint16_t*)mine);
  auto dma = [&](int ks, int st) {
    const uint32_t l0 = lmine + st * SLICE * 2;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      lds_dma16(pa[u] + (int64_t)ks * ka, l0 + u * 1024);
      lds_dma16(pb[u] + (int64_t)ks * kb, l0 + KW * BM * 2 + u * 1024);
    }
  };
  // fragments: lane (tg, tq, tc) reads slice rows 8 tg + tq (+ 4) at column
  // 4 tc of each 16-column block (see tr_frag)
  const int tg = lane >> 4, tq = (lane & 15) >> 2, tc = lane & 3;
  const int trow = 8 * tg + tq, hp = kperm8(trow);
  int fo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) fo[i] = trow * BM + (((2 * i) + (tc >> 1)) ^ hp) * 8 + (tc & 1) * 4;

  // k-steps whose rows of this wave's slice exist: the first nkw
  const int nkw = K > KW * wv ? (K - KW * wv + BK - 1) / BK : 0;
  if (nkw > 0) dma(0, 0);
  for (int j = 0; j < nkw; ++j) {
    // the other slice was last read by k-step j - 1, whose reads completed
    // before its MFMAs were issued
    if (j + 1 < nkw) {
      dma(j + 1, (j + 1) & 1);
      asm volatile("s_waitcnt vmcnt(8)" ::: "memory");  // k-step j's eight loads have landed
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    const uint16_t* st = mine + (j & 1) * SLICE;
    u32x4_t fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = tr_frag(st + fo[i], BM);
#pragma unroll
    for (int i = 0; i < 4; ++i) fb[i] = tr_frag(st + KW * BM + fo[i], BN);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[i]),
                                                             __builtin_bit_cast(bf16x8_t, fb[jj]), acc[i][jj], 0, 0, 0);
    if (do_rows) {
#pragma unroll
      for (int i = 0; i < 4; ++i) rs[i] += sum8_bf16(fa[i]);
    }
  }

  // Adam items: rows (tid >> 4) + 16 it, columns 4 (tid & 15) of the tile.
  // The parameters and moments are loaded now, while the partial tiles are
  // added (loaded before the main loop they would hold 48 registers through
  // it).
  typedef float f32x4a_t __attribute__((ext_vector_type(4), aligned(4)));
  typedef __attribute__((address_space(1))) f32x4a_t gvec;
  const int ac = 4 * (tid & 15);
  f32x4a_t apv[IT], amv[IT], avv[IT];
  bool afull[IT];
  int64_t afi[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int m = m0 + (tid >> 4) + 16 * it, n = n0 + ac;
    afull[it] = m < g.M && n + 4 <= g.N;
    afi[it] = (int64_t)m * g.N + n;
    if (afull[it]) {
      apv[it] = *reinterpret_cast<const gvec*>(gmem(e.ap) + afi[it]);
      amv[it] = *reinterpret_cast<const gvec*>(gmem(e.am) + afi[it]);
      avv[it] = *reinterpret_cast<const gvec*>(gmem(e.av) + afi[it]);
    }
  }

  // Partial tiles through LDS, row-major with the 16-column blocks of row r
  // permuted by 16 ((r >> 2) & 3) (conflict-free stores); the bias row sums
  // of the waves into a buffer of their own.
  float* red = reinterpret_cast<float*>(smem);
  float* rsum = reinterpret_cast<float*>(smem + MAIN);
  if (do_rows) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float sr = rs[i];
      sr += __shfl_xor(sr, 16, 64);
      sr += __shfl_xor(sr, 32, 64);
      if (lane < 16) rsum[wv * BM + 16 * i + lane] = sr;
    }
  }
  __syncthreads();  // every wave is done with its slices
  {
    float* rw = red + wv * BM * BN;
    const int sw = 16 * tg;  // rows 16 i + 4 tg + q: (r >> 2) & 3 == tg
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int q = 0; q < 4; ++q) rw[(16 * i + 4 * tg + q) * BN + ((16 * jj + (lane & 15)) ^ sw)] = acc[i][jj][q];
  }
  __syncthreads();
  f32x4_t gv[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int r = (tid >> 4) + 16 * it;
    const float* src = red + r * BN + (ac ^ (16 * ((r >> 2) & 3)));
    gv[it] = *reinterpret_cast<const f32x4_t*>(src);
#pragma unroll
    for (int w = 1; w < NW; ++w) gv[it] += *reinterpret_cast<const f32x4_t*>(src + w * BM * BN);
  }
  const float step = e.hyper[0], bc2s = e.hyper[1];
  if (do_rows && tid < BM && m0 + tid < g.M) {
    float sr = rsum[tid];
#pragma unroll
    for (int w = 1; w < NW; ++w) sr += rsum[w * BM + tid];
    const int m = m0 + tid;
    if (e.bp) {
      // the bias's Adam update: this tile holds its rows' whole gradient
      float p = e.bp[m], mo = e.bm[m], v = e.bv[m];
      adam_elem(p, mo, v, sr, e.b1, e.b2, step, bc2s, e.eps);
      if (e.bg) e.bg[m] = sr;
      e.bm[m] = mo;
      e.bv[m] = v;
      e.bp[m] = p;
    } else {
      e.bpart[m] = sr;
    }
  }
  // Adam of the tile's parameters: items of 4 consecutive columns of one row
  // (16-byte accesses at 4-byte alignment: parameter rows start anywhere);
  // a row's ragged end goes element by element
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int m = m0 + (tid >> 4) + 16 * it, n = n0 + ac;
    if (afull[it]) {
      float pp[4], mm[4], vq[4];
      uint16_t o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        pp[k] = apv[it][k];
        mm[k] = amv[it][k];
        vq[k] = avv[it][k];
        adam_elem(pp[k], mm[k], vq[k], gv[it][k], e.b1, e.b2, step, bc2s, e.eps);
        o[k] = f2bf(pp[k]);
      }
      if (e.ag)
        __builtin_nontemporal_store(f32x4a_t{gv[it][0], gv[it][1], gv[it][2], gv[it][3]},
                                    reinterpret_cast<gvec*>(gmem(e.ag) + afi[it]));
      __builtin_nontemporal_store(f32x4a_t{mm[0], mm[1], mm[2], mm[3]}, reinterpret_cast<gvec*>(gmem(e.am) + afi[it]));
      __builtin_nontemporal_store(f32x4a_t{vq[0], vq[1], vq[2], vq[3]}, reinterpret_cast<gvec*>(gmem(e.av) + afi[it]));
      __builtin_nontemporal_store(f32x4a_t{pp[0], pp[1], pp[2], pp[3]}, reinterpret_cast<gvec*>(gmem(e.ap) + afi[it]));
      st4(static_cast<uint16_t*>(e.ash) + (int64_t)m * e.ldash + n, o);  // copy rows: 64-element multiples
    } else if (m < g.M && n < g.N) {
      for (int k = 0; k < g.N - n && k < 4; ++k) {
        const float gk = gv[it][k];
        float pp = e.ap[afi[it] + k], mm = e.am[afi[it] + k], vq = e.av[afi[it] + k];
        adam_elem(pp, mm, vq, gk, e.b1, e.b2, step, bc2s, e.eps);
        if (e.ag) e.ag[afi[it] + k] = gk;
        e.am[afi[it] + k] = mm;
        e.av[afi[it] + k] = vq;
        e.ap[afi[it] + k] = pp;
        static_cast<uint16_t*>(e.ash)[(int64_t)m * e.ldash + n + k] = f2bf(pp);
      }
    }
  }
}

__global__ __launch_bounds__(256) void erase_wgrad_adam_w4(GemmDesc g, EpiParams e, AdamArgs a, int ntiles) {
  __shared__ __attribute__((aligned(16))) char smem[w4::BYTES];
  static_assert(w4::BYTES >= ADAM_TR * ADAM_TC * 2, "staging");
  const int b = blockIdx.x;
  if (b < ntiles) {
    const TileIdx ti = tile_from(xcd_linear(b, ntiles), (g.M + 63) / 64, (g.N + 63) / 64, g.group);
    wgrad_adam_w4_tile(g, e, ti.m, ti.n, smem);
  } else {
    uint16_t(*s_o)[ADAM_TC] = reinterpret_cast<uint16_t(*)[ADAM_TC]>(smem);
    adam_chunk<uint16_t>(a, b - ntiles, (int)threadIdx.x, s_o);
  }
}

static hipError_t launch_wgrad_w8(const GemmDesc& g0, const EpiParams& e, const AdamArgs& a, hipStream_t s,
                                  const LaunchEv& ev) {
  if (g0.K % 64 != 0) return hipErrorInvalidValue;  // whole 32-row slices
  const GemmDesc g = with_group(g0, 64, 64);
  const int ntiles = ((g.M + 63) / 64) * ((g.N + 63) / 64);
  const dim3 grid((unsigned)(ntiles + a.nchunks)), block(256);
  ERASE_LAUNCH(erase_wgrad_adam_w4, grid, block, 0, s, ev, g, e, a, ntiles);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Vocabulary logits in wide tiles (bf16): e[m][n] = exp(sum_k h[m][k] w[n][k]
// - xref[m]) rounded to bf16, and per row and 128-column tile the sum of the
// stored values (the epilogue of GK_FWD_LOGITS).  A workgroup of eight waves
// computes 256 positions x 256 vocabulary rows, each wave 64 x 128, so a
// wave reads 24 KB of MFMA fragments from LDS per 64 x 128 x 64 slab (the
// GEMM core's 2 x 2 waves of 32 x 64 read 12 KB per slab of a quarter of
// that work), and the operands cross L2 once per 256 x 256 tile.  The
// operand rows of a 64-wide k-step (one 128-byte line per row) go straight
// from global memory into one of two 64 KB LDS stages
// (global_load_lds_dwordx4; chunk c of row r at slot c ^ (r & 7):
// conflict-free 16-byte fragment reads), the next k-step in flight, one
// barrier per k-step; two waves per SIMD.  The workgroups are persistent
// (one per CU: the stages leave no room for a second), and each loads the
// first k-step of its next tile during the last k-step of the current one.
// Measured at 16384 x 32768 x 512 (kernel alone, one MI355X): 761-766 us
// against 834 us for one workgroup per tile (whose first k-step waited for
// its loads) and 807 us for that form in groups of two M-tiles; on another
// MI355X the one-tile form took 818-821 us against 857-881 us for a 128 x 256
// form (four waves, 32-wide k-steps in three 24 KB stages, two workgroups
// per CU: each operand line fetched in two halves) and about 1 ms for the
// GEMM core's 64 x 128 tiles.  The MFMA computes the transposed
// tile (vocabulary rows as the A operand): a lane holds 4 consecutive
// vocabulary columns of one position, stored as 8 bytes; a row's sum over a
// 128-column tile adds the lane's 32 values, then the 4 lane groups, in a
// fixed order.
// ---------------------------------------------------------------------------
namespace lgw {
constexpr int BM = 256, BN = 256, BK = 64;  // positions, vocabulary rows per workgroup; k-step
constexpr int NW = 8, NT = 64 * NW;         // waves and threads
constexpr int NST = 2;                      // LDS stages
constexpr int STAGE = (BM + BN) * BK * 2;   // 64 KB: rows of 128 bytes
constexpr int LOADS = (BM + BN) / 8 / NW;   // loads of 8 rows per wave and k-step
// M-tiles per group of the tile order (each group walks every vocabulary
// tile): two, so the 32 tiles an XCD runs at once read 2 position blocks
// and 16 vocabulary blocks (persistent form, one MI355X: groups of 1, 2, 4,
// 8, 16 took 795-798, 761-766, 772-779, 790, 783 us)
constexpr int GROUP = 2;
}  // namespace lgw

__global__ __launch_bounds__(lgw::NT) void erase_fwd_logits_wide(GemmDesc g, EpiParams e) {
  using namespace lgw;
  // two operand stages, then two 1 KB slots of reference logits (one tile's
  // 256 positions each, alternating between consecutive tiles)
  __shared__ __attribute__((aligned(16))) char smem[NST * STAGE + 2 * BM * 4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv & 3, wn = wv >> 2;  // the wave's 64 positions and 128 vocabulary rows
  const int gm = g.M / BM, gn = g.N / BN, ntiles = gm * gn;
  const int nk = g.K / BK;
  const int fr = lane & 15, fg = lane >> 4;
  constexpr float kL2e = 1.4426950408889634f;

  // Kernel arguments in registers: the loads' asm statements clobber memory,
  // so values read from the arguments inside the loops would be loaded
  // again (scalar loads and a full wait) before every load.  Row strides of
  // 8 rows for the direct-to-LDS loads.
  const int64_t lda = g.lda, ldb = g.ldb, sa = 8 * lda, sw = 8 * ldb, ldy = e.ldy, ldls = e.ldlstat;
  uint16_t* Y = static_cast<uint16_t*>(e.y);
  float* lstat = e.lstat;
  // direct-to-LDS loads: load u of wave wv fills stage rows 8 ui .. 8 ui + 7,
  // ui = LOADS wv + u (rows [0, BM) positions, then vocabulary rows); lane l
  // writes row 8 ui + (l >> 3), slot l & 7, which holds chunk (l & 7) ^ (l >> 3).
  // A wave's loads all read one operand: the first BM / (8 LOADS) waves the
  // positions, the others the vocabulary rows.  The addresses are a
  // wave-uniform base (scalar registers) plus the lane's fixed byte offset.
  static_assert((BM / 8) % LOADS == 0, "a wave's loads read one operand");
  const bool wa = wv < BM / (8 * LOADS);
  const int ch = (lane & 7) ^ (lane >> 3);
  const uint32_t voff = (uint32_t)((lane >> 3) * (wa ? lda : ldb) * 2 + ch * 16);
  const int64_t rstride = (wa ? sa : sw) * 2;  // bytes between a wave's 8-row groups
  const int r0 = 8 * (wa ? LOADS * wv : LOADS * wv - BM / 8);  // the wave's first row of its operand
  const char* Ab = static_cast<const char*>(g.A) + (int64_t)r0 * lda * 2;
  const char* Wb = static_cast<const char*>(g.B) + (int64_t)r0 * ldb * 2;
  const char* Xb = reinterpret_cast<const char*>(e.xref);
  const uint32_t lbase = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) char*)smem);
  const uint32_t lwave = lbase + LOADS * wv * 1024;
  const float* sxr = reinterpret_cast<const float*>(smem + NST * STAGE);
  auto dma = [&](int64_t oa, int64_t ow, int ks, int st) {
    const char* b = (wa ? Ab + oa * 2 : Wb + ow * 2) + ks * BK * 2;
    const uint32_t l0 = lwave + st * STAGE;
#pragma unroll
    for (int u = 0; u < LOADS; ++u) lds_dma16s(b + u * rstride, voff, l0 + u * 1024);
  };
  // a tile's 256 reference logits into its slot: one load by wave 0
  auto dma_xref = [&](int m0, int slot) {
    if (wv == 0) lds_dma16s(Xb + (int64_t)m0 * 4, 16 * lane, lbase + NST * STAGE + slot * BM * 4);
  };

  // fragment reads: row block at stage row R0 (a multiple of 16), k half h:
  // lane reads row R0 + (l & 15), chunk 4 h + (l >> 4), at slot chunk ^ (l & 7)
  const int fo0 = fr * 128 + ((0 + fg) ^ (lane & 7)) * 16, fo1 = fr * 128 + ((4 + fg) ^ (lane & 7)) * 16;

  // Persistent workgroups: workgroup b runs tiles b, b + G, b + 2G, ... (G
  // the grid, a multiple of the XCD count, so every tile of a workgroup lies
  // in its own XCD's range).  The first k-step of the next tile and its
  // reference logits are loaded during the last k-step of the current one,
  // so their latency hides behind that k-step's MFMAs and the epilogue.
  const int G = (int)gridDim.x;
  int t = (int)blockIdx.x;
  if (t >= ntiles || nk <= 0) return;
  TileIdx ti = tile_from(xcd_linear(t, ntiles), gm, gn, GROUP);
  int64_t oa = (int64_t)(ti.m * BM) * lda, ow = (int64_t)(ti.n * BN) * ldb;
  dma_xref(ti.m * BM, 0);
  dma(oa, ow, 0, 0);
  int st0 = 0, slot = 0;  // the stage of the tile's first k-step; its reference-logit slot
  bool first = true;
  for (;;) {
    const int m0 = ti.m * BM, n0 = ti.n * BN;
    const int tn = t + G;
    const bool more = tn < ntiles;
    TileIdx tin = ti;
    if (more) tin = tile_from(xcd_linear(tn, ntiles), gm, gn, GROUP);
    const int64_t oan = (int64_t)(tin.m * BM) * lda, own = (int64_t)(tin.n * BN) * ldb;

    f32x4_t acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int ks = 0; ks < nk; ++ks) {
      // this wave's loads of k-step ks have landed; after the barrier every
      // wave's have, and every wave is done reading k-step ks - 1, whose
      // stage the next loads overwrite.  The first k-step of a later tile
      // was loaded before the previous tile's epilogue, whose 36 stores (32
      // of the exponentials, 4 of the row sums) were issued after it: the
      // counter at 32 means it has landed.
      if (ks == 0 && !first)
        asm volatile("s_waitcnt vmcnt(32)" ::: "memory");
      else
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (ks + 1 < nk) {
        dma(oa, ow, ks + 1, (st0 + ks + 1) % NST);
      } else if (more) {
        dma_xref(tin.m * BM, slot ^ 1);
        dma(oan, own, 0, (st0 + nk) % NST);
      }
      const char* st = smem + ((st0 + ks) % NST) * STAGE;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int fo = h ? fo1 : fo0;
        u32x4_t fw[8], fh[4];
#pragma unroll
        for (int i = 0; i < 8; ++i)
          fw[i] = *reinterpret_cast<const u32x4_t*>(st + (BM + 128 * wn + 16 * i) * 128 + fo);
#pragma unroll
        for (int j = 0; j < 4; ++j) fh[j] = *reinterpret_cast<const u32x4_t*>(st + (64 * wm + 16 * j) * 128 + fo);
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fw[i]),
                                                                __builtin_bit_cast(bf16x8_t, fh[j]), acc[i][j], 0, 0, 0);
      }
    }

    // acc[i][j][q]: vocabulary row n0 + 128 wn + 16 i + 4 (l >> 4) + q of
    // position m0 + 64 wm + 16 j + (l & 15)
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const int tcol = (n0 + 128 * wn) / 128;  // the row-sum tile
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int pl = 64 * wm + 16 * j + fr, p = m0 + pl;
      const float xl = sxr[slot * BM + pl] * kL2e;
      float se = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float ev[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) ev[q] = __builtin_amdgcn_exp2f(fmaf(acc[i][j][q], kL2e, -xl));
        const uint32_t o0 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{ev[0], ev[1]}), bf16x2_t));
        const uint32_t o1 = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{ev[2], ev[3]}), bf16x2_t));
        se += __uint_as_float(o0 << 16);
        se += __uint_as_float(o0 & 0xffff0000u);
        se += __uint_as_float(o1 << 16);
        se += __uint_as_float(o1 & 0xffff0000u);
        *reinterpret_cast<uint2*>(Y + (int64_t)p * ldy + n0 + 128 * wn + 16 * i + 4 * fg) = uint2{o0, o1};
      }
      se += __shfl_xor(se, 16, 64);
      se += __shfl_xor(se, 32, 64);
      if (fg == 0) lstat[(int64_t)p * ldls + tcol] = se;
    }
    if (!more) break;
    t = tn;
    ti = tin;
    oa = oan;
    ow = own;
    st0 = (st0 + nk) % NST;
    slot ^= 1;
    first = false;
  }
}

static bool logits_wide_fits(const GemmDesc& g, const EpiParams& e) {
  // whole 256 x 256 tiles and 64-wide k-steps within both operand rows;
  // 8-byte output stores; reference logits in 16-byte chunks
  return g.split == 1 && g.M > 0 && g.M % lgw::BM == 0 && g.N % lgw::BN == 0 && g.K % lgw::BK == 0 && g.K > 0 &&
         g.K <= g.lda && g.K <= g.ldb && e.ldy % 4 == 0 && (reinterpret_cast<uintptr_t>(e.y) & 7) == 0 &&
         (reinterpret_cast<uintptr_t>(e.xref) & 15) == 0;
}

// Compute units of the current device (cached per device).
static int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64 && cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  if (dev < 64) cached[dev] = n;
  return n;
}

static hipError_t launch_logits_wide(const GemmDesc& g, const EpiParams& e, hipStream_t s, const LaunchEv& ev) {
  // one persistent workgroup per compute unit (the 128 KB of stages allow
  // no second), a multiple of the XCD count
  const int tiles = (g.M / lgw::BM) * (g.N / lgw::BN);
  int grid = std::max(kXcds, device_cus() / kXcds * kXcds);
  if (grid > tiles) grid = tiles;
  ERASE_LAUNCH(erase_fwd_logits_wide, dim3((unsigned)grid), dim3(lgw::NT), 0, s, ev, g, e);
  return hipGetLastError();
}

hipError_t launch_wgrad_adam(int bf16, const GemmDesc& g0, const EpiParams& e, const AdamArgs& a, hipStream_t s,
                             const LaunchEv& ev) {
  if (g0.bm != 64 || g0.bn != 64 || g0.kgroups != 2 || g0.split != 1 || !e.ap) return hipErrorInvalidValue;
  if (bf16) return launch_wgrad_w8(g0, e, a, s, ev);
  const GemmDesc g = with_group(g0, 64, 64);
  const int ntiles = ((g.M + 63) / 64) * ((g.N + 63) / 64);
  const dim3 grid((unsigned)(ntiles + (a.nchunks + 1) / 2)), block(512);
  ERASE_LAUNCH((erase_wgrad_adam_kg2<float, 64, 64>), grid, block, 0, s, ev, g, e, a, ntiles);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void erase_refresh(AdamArgs a) {
  const int64_t chunk = blockIdx.x;
  const AdamSeg sg = a.seg[find_seg(a, chunk)];
  const int tile = (int)(chunk - sg.chunk0);
  const int r0 = (tile / sg.tcols) * ADAM_TR;
  const int c = (tile % sg.tcols) * ADAM_TC + (int)threadIdx.x;
  if ((int)threadIdx.x >= ADAM_TC || c >= sg.cols) return;
  for (int q = 0; q < ADAM_TR && r0 + q < sg.rows; ++q) {
    const int r = r0 + q;
    const float p = gmem(sg.p)[(int64_t)r * sg.cols + c];
    if (sg.sh) gmem(static_cast<T*>(sg.sh))[(int64_t)r * sg.ldsh + c] = cvt<T>(p);
    if (sg.sht) gmem(static_cast<T*>(sg.sht))[(int64_t)c * sg.ldsht + r] = cvt<T>(p);
  }
}

hipError_t launch_adam(int bf16, const AdamArgs& a, hipStream_t s, const LaunchEv& ev) {
  dim3 grid((unsigned)a.nchunks), block(256);
  if (bf16)
    ERASE_LAUNCH(erase_adam<uint16_t>, grid, block, 0, s, ev, a);
  else
    ERASE_LAUNCH(erase_adam<float>, grid, block, 0, s, ev, a);
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
