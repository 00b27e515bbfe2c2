// HIP kernels of the detached small-transformer step (gfx950, bf16 storage,
// fp32 arithmetic).  The projections, the MLP and the vocabulary head are GEMMs
// of the shared GEMM core (kernels.hip); this file holds the rest:
//
//  * tf_embed:      a0[n] = E[token n] from the bf16 copy of the embedding,
//                   and the next-token target of every position.
//  * tf_rms_fwd:    y = x r with r = 1 / sqrt(mean(x^2) + eps) per row.
//  * tf_rms_bwd:    dx = r (dy - y mean(dy y)) (+ a residual gradient).
//  * tf_attn_fwd:   causal softmax attention of every head (head size 64),
//                   online over key blocks of 64 (the next block's loads in
//                   flight during the current one); o and the row
//                   log-sum-exp.
//  * tf_attn_bwd_*: D = rowsum(do * o), then dK/dV per key block and dQ per
//                   query block (no atomics: every output has one writer).
//  * tf_head_norm:  the softmax normaliser of every row from the logits
//                   GEMM's per-tile sums of exponentials relative to the
//                   target logit: the row loss, the row's gradient scale,
//                   the target entry of the gradient and the scaled head
//                   input; tf_head_fix recomputes the rare rows whose
//                   exponentials were out of range.
//  * tf_emb_*:      embedding gradient: positions bucketed by token (integer
//                   counters), each bucket ordered by position, rows summed in
//                   that order, so the result does not depend on scheduling.
//
// MFMA v_mfma_f32_16x16x32_bf16 operand layout (lane l, g = l >> 4):
//   A: A[m = l & 15][k = 8g .. 8g + 7];  B: B[k = 8g .. 8g + 7][n = l & 15];
//   C: C[m = 4g + q][n = l & 15], q = 0..3.
// Attention computes S^T = K Q^T with the key rows of the A operand
// permuted, row r of sub-tile t being key 8 (r >> 2) + 4 t + (r & 3); lane l
// then holds, for query row l & 15, the scores of keys 8g + 4t + q, i.e. the
// 8 consecutive keys 8g .. 8g + 7 over t = 0, 1: exactly the B operand of
// O^T = V^T P^T.  Softmax statistics are per lane (one query row) and the
// output accumulator O^T is rescaled per lane.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace erase {

#define ERASE_TF_LAUNCH(KERNEL, GRID, BLOCK, STREAM, EV, ARG)                              \
  do {                                                                                   \
    if ((EV).e0)                                                                         \
      hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, 0, STREAM, (EV).e0, (EV).e1, 0, ARG);  \
    else                                                                                 \
      hipLaunchKernelGGL(KERNEL, GRID, BLOCK, 0, STREAM, ARG);                           \
  } while (0)

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ uint16_t tobf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t pack2(float a, float b) { return (uint32_t)tobf(a) | ((uint32_t)tobf(b) << 16); }
__device__ __forceinline__ float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ f32x4_t mfma(const u32x4_t& a, const u32x4_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

// ---------------------------------------------------------------------------
// LDS tiles of 64 rows x 64 bf16 (128-byte rows); 16-byte chunk c of row r is
// stored at chunk c ^ (r & 7)
// ---------------------------------------------------------------------------
__device__ __forceinline__ int tix(int r, int col) { return r * 64 + (((col >> 3) ^ (r & 7)) << 3) + (col & 7); }

// 8 consecutive elements of row r starting at column 8 c (one chunk)
__device__ __forceinline__ u32x4_t row_chunk(const uint16_t* t, int r, int c) {
  return *reinterpret_cast<const u32x4_t*>(t + r * 64 + ((c ^ (r & 7)) << 3));
}

// MFMA operand of 8 consecutive rows r0 + 8g .. r0 + 8g + 7 at column
// c16 + (l & 15): two transposing 8-byte reads (each lane names 4 elements
// of row r0 + 8g + ((l & 15) >> 2) (+ 4) at column c16 + 4 (l & 3); lane l
// receives element l & 3 of the reads of lanes 4q + (l >> 2) of its 16-lane
// group, q = 0..3).
__device__ __forceinline__ u32x4_t col_frag(const uint16_t* t, int r0, int c16, int lane) {
  typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;
  const int r = r0 + 8 * (lane >> 4) + ((lane & 15) >> 2);
  const int col = c16 + 4 * (lane & 3);
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(t + tix(r, col)));
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(t + tix(r + 4, col)));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return u32x4_t{a.x, a.y, b.x, b.y};
}

// Staging of rows [row0, row0 + 64), columns [col0, col0 + 64) of a bf16
// matrix into an LDS tile by 256 threads (rows at or past `rows` are zero),
// in two halves: the thread's two chunks into registers, then into the
// tile, so the loads of the next block are in flight while the current one
// is computed.
struct Stage2 {
  u32x4_t v[2];
};
__device__ __forceinline__ Stage2 load64(const uint16_t* g, int64_t ld, int row0, int rows, int64_t col0, int tid) {
  Stage2 r;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + 256 * i;
    const int rr = c >> 3, ch = c & 7;
    r.v[i] = u32x4_t{0u, 0u, 0u, 0u};
    if (row0 + rr < rows) r.v[i] = *reinterpret_cast<const u32x4_t*>(g + (int64_t)(row0 + rr) * ld + col0 + ch * 8);
  }
  return r;
}
__device__ __forceinline__ void store64(uint16_t* t, const Stage2& r, int tid) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + 256 * i;
    const int rr = c >> 3, ch = c & 7;
    *reinterpret_cast<u32x4_t*>(t + rr * 64 + ((ch ^ (rr & 7)) << 3)) = r.v[i];
  }
}

// Row of the permuted A operand: sub-tile t, lane l -> local row
// 8 ((l & 15) >> 2) + 4 t + (l & 3) within a 32-row half
__device__ __forceinline__ int prow(int lane, int t) { return 8 * ((lane & 15) >> 2) + 4 * t + (lane & 3); }

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace

// ---------------------------------------------------------------------------
// embedding gather and targets
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void tf_embed(TfEmbedArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + wave;
  if (n >= (int64_t)a.B * a.T) return;
  const int b = (int)(n / a.T), t = (int)(n % a.T);
  const int32_t tok = a.tokens[(int64_t)b * (a.T + 1) + t];
  const int32_t nxt = a.tokens[(int64_t)b * (a.T + 1) + t + 1];
  const bool ok = tok >= 0 && tok < a.V;
  if (lane == 0) {
    a.target[n] = (nxt >= 0 && nxt < a.V) ? nxt : -1;
    a.input[n] = ok ? tok : -1;
    if (!ok || !(nxt >= 0 && nxt < a.V)) a.status[0] = 2;
  }
  for (int c = lane; c < a.d / 8; c += 64) {
    u32x4_t v = {0u, 0u, 0u, 0u};
    if (ok) v = *reinterpret_cast<const u32x4_t*>(a.emb + (int64_t)tok * a.ldemb + c * 8);
    *reinterpret_cast<u32x4_t*>(a.a0 + n * a.lda0 + c * 8) = v;
  }
}

// ---------------------------------------------------------------------------
// RMSNorm forward / backward: one wave per row, row width d (multiple of 8,
// at most 4096), 16-byte chunks
// ---------------------------------------------------------------------------
constexpr int kRmsChunks = 8;  // chunks per lane: d <= 64 * 8 * 8

__global__ __launch_bounds__(256) void tf_rms_fwd(TfRmsArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + wave;
  if (n >= a.N) return;
  const int nc = a.d / 8;
  u32x4_t v[kRmsChunks];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kRmsChunks; ++i) {
    const int c = lane + 64 * i;
    v[i] = u32x4_t{0u, 0u, 0u, 0u};
    if (c < nc) v[i] = *reinterpret_cast<const u32x4_t*>(a.x + n * a.ldx + c * 8);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float x0 = lo16(v[i][k]), x1 = hi16(v[i][k]);
      ss = fmaf(x0, x0, ss);
      ss = fmaf(x1, x1, ss);
    }
  }
  ss = wsum(ss);
  const float r = 1.f / sqrtf(ss / (float)a.d + a.eps);
  if (lane == 0) a.r[n] = r;
  const int32_t tg = a.hw ? a.target[n] : -1;
  float xt = 0.f;
#pragma unroll
  for (int i = 0; i < kRmsChunks; ++i) {
    const int c = lane + 64 * i;
    if (c >= nc) continue;
    u32x4_t o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = pack2(lo16(v[i][k]) * r, hi16(v[i][k]) * r);
    *reinterpret_cast<u32x4_t*>(a.y + n * a.ldy + c * 8) = o;
    if (tg >= 0) {
      // the target logit of the stored (rounded) row
      const u32x4_t w = *reinterpret_cast<const u32x4_t*>(a.hw + (int64_t)tg * a.ldhw + c * 8);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        xt = fmaf(lo16(o[k]), lo16(w[k]), xt);
        xt = fmaf(hi16(o[k]), hi16(w[k]), xt);
      }
    }
  }
  if (a.hw) {
    xt = wsum(xt);
    if (lane == 0) a.xref[n] = xt;
  }
}

__global__ __launch_bounds__(256) void tf_rms_bwd(TfRmsArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + wave;
  if (n >= a.N) return;
  const int nc = a.d / 8;
  const float r = a.r[n];
  const float gs = a.dyscale ? a.dyscale[n] : 1.f;
  u32x4_t xv[kRmsChunks], gv[kRmsChunks];
  float dot = 0.f;
#pragma unroll
  for (int i = 0; i < kRmsChunks; ++i) {
    const int c = lane + 64 * i;
    xv[i] = gv[i] = u32x4_t{0u, 0u, 0u, 0u};
    if (c < nc) {
      xv[i] = *reinterpret_cast<const u32x4_t*>(a.x + n * a.ldx + c * 8);
      gv[i] = *reinterpret_cast<const u32x4_t*>(a.dy + n * a.lddy + c * 8);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      dot = fmaf(lo16(gv[i][k]) * gs, lo16(xv[i][k]) * r, dot);
      dot = fmaf(hi16(gv[i][k]) * gs, hi16(xv[i][k]) * r, dot);
    }
  }
  const float mdot = wsum(dot) / (float)a.d;
#pragma unroll
  for (int i = 0; i < kRmsChunks; ++i) {
    const int c = lane + 64 * i;
    if (c >= nc) continue;
    float o[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      o[2 * k] = r * (lo16(gv[i][k]) * gs - lo16(xv[i][k]) * r * mdot);
      o[2 * k + 1] = r * (hi16(gv[i][k]) * gs - hi16(xv[i][k]) * r * mdot);
    }
    if (a.res) {
      const u32x4_t rv = *reinterpret_cast<const u32x4_t*>(a.res + n * a.ldres + c * 8);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        o[2 * k] += lo16(rv[k]);
        o[2 * k + 1] += hi16(rv[k]);
      }
    }
    if (a.out_f32) {
      float* dst = a.out_f32 + n * a.ldout + c * 8;
      *reinterpret_cast<float4*>(dst) = make_float4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(o[4], o[5], o[6], o[7]);
    } else {
      u32x4_t w;
#pragma unroll
      for (int k = 0; k < 4; ++k) w[k] = pack2(o[2 * k], o[2 * k + 1]);
      *reinterpret_cast<u32x4_t*>(a.y + n * a.ldy + c * 8) = w;
    }
  }
}

// ---------------------------------------------------------------------------
// attention forward: workgroup = (query block of 64, head, sequence), wave w
// owns query rows q0 + 16 w + (l & 15)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void tf_attn_fwd(TfAttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sk[64 * 64];
  __shared__ __attribute__((aligned(16))) uint16_t sv[64 * 64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4;
  const int nqb = (a.T + 63) / 64;
  const int qb = nqb - 1 - (int)blockIdx.x;  // the longest rows first
  const int h = blockIdx.y, b = blockIdx.z;
  const int q0 = qb * 64;
  const int qrow = q0 + 16 * wave + (lane & 15);
  const int64_t base = (int64_t)b * a.T;
  const int64_t colq = (int64_t)h * 64, colk = a.d + colq, colv = 2 * (int64_t)a.d + colq;
  // B operand of S^T = K Q^T: Q[qrow][32 s + 8 g .. + 7]
  u32x4_t qf[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    qf[s] = u32x4_t{0u, 0u, 0u, 0u};
    if (qrow < a.T) qf[s] = *reinterpret_cast<const u32x4_t*>(a.qkv + (base + qrow) * a.ldqkv + colq + 32 * s + 8 * g);
  }
  const float sc = a.scale * kLog2e;  // scores in log2 units
  float mrow = -1e30f, lpart = 0.f;
  f32x4_t ot[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) ot[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const uint16_t* kvbase = a.qkv + base * a.ldqkv;
  Stage2 nk = load64(kvbase, a.ldqkv, 0, a.T, colk, tid), nv = load64(kvbase, a.ldqkv, 0, a.T, colv, tid);
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * 64;
    __syncthreads();  // previous block's reads done
    store64(sk, nk, tid);
    store64(sv, nv, tid);
    __syncthreads();
    if (kb < qb) {  // next block's loads in flight during this block's compute
      nk = load64(kvbase, a.ldqkv, k0 + 64, a.T, colk, tid);
      nv = load64(kvbase, a.ldqkv, k0 + 64, a.T, colv, tid);
    }
    // scores of keys k0 + 32 st + 8 g + 4 t + q
    f32x4_t st4[2][2];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        st4[st][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int kr = 32 * st + prow(lane, t);
#pragma unroll
        for (int s = 0; s < 2; ++s) st4[st][t] = mfma(row_chunk(sk, kr, 4 * s + g), qf[s], st4[st][t]);
      }
    float mb = -1e30f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int key = k0 + 32 * st + 8 * g + 4 * t + q;
          const bool ok = key <= qrow && key < a.T;
          const float v = ok ? st4[st][t][q] * sc : -INFINITY;
          st4[st][t][q] = v;
          mb = fmaxf(mb, v);
        }
    mb = fmaxf(mb, __shfl_xor(mb, 16, 64));
    mb = fmaxf(mb, __shfl_xor(mb, 32, 64));
    const float mnew = fmaxf(mrow, mb);
    const float alpha = __builtin_amdgcn_exp2f(mrow - mnew);
    mrow = mnew;
    lpart *= alpha;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) ot[dt] *= alpha;
    u32x4_t pf[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      float p[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          p[4 * t + q] = __builtin_amdgcn_exp2f(st4[st][t][q] - mnew);
          lpart += p[4 * t + q];
        }
      pf[st] = u32x4_t{pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
    }
    // O^T[dh][qrow] += V^T[dh][key] P^T[key][qrow]
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int st = 0; st < 2; ++st) ot[dt] = mfma(col_frag(sv, 32 * st, 16 * dt, lane), pf[st], ot[dt]);
  }
  float l = lpart + __shfl_xor(lpart, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (qrow < a.T) {
    const float inv = 1.f / l;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      uint2 w;
      w.x = pack2(ot[dt][0] * inv, ot[dt][1] * inv);
      w.y = pack2(ot[dt][2] * inv, ot[dt][3] * inv);
      *reinterpret_cast<uint2*>(a.o + (base + qrow) * a.ldo + colq + 16 * dt + 4 * g) = w;
    }
    if (g == 0) a.lse[((int64_t)b * a.H + h) * a.T + qrow] = (mrow + log2f(l)) * kLn2;
  }
}

// D[b][h][t] = sum over the head's 64 columns of do * o: 8 lanes per row
__global__ __launch_bounds__(256) void tf_attn_bwd_pre(TfAttnArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 32 + (threadIdx.x >> 3);  // (position, head)
  const int j = threadIdx.x & 7;
  const int64_t n = i / a.H;
  const int h = (int)(i % a.H);
  float s = 0.f;
  if (n < (int64_t)a.B * a.T) {
    const u32x4_t x = *reinterpret_cast<const u32x4_t*>(a.o + n * a.ldo + h * 64 + 8 * j);
    const u32x4_t y = *reinterpret_cast<const u32x4_t*>(a.dout + n * a.lddo + h * 64 + 8 * j);
#pragma unroll
    for (int k = 0; k < 4; ++k) s += lo16(x[k]) * lo16(y[k]) + hi16(x[k]) * hi16(y[k]);
  }
  s += __shfl_xor(s, 1, 64);
  s += __shfl_xor(s, 2, 64);
  s += __shfl_xor(s, 4, 64);
  if (j == 0 && n < (int64_t)a.B * a.T) {
    const int b = (int)(n / a.T), t = (int)(n % a.T);
    a.dsum[((int64_t)b * a.H + h) * a.T + t] = s;
  }
}

// dK, dV of a key block: wave w owns keys k0 + 16 w + (l & 15); for every
// query block at or after the key block, S = Q K^T and dP = dO V^T with the
// query rows of the A operand permuted, so lane l holds, for its key, query
// rows 8g .. 8g + 7 of each 32-row half: the B operand of dV^T = dO^T P and
// dK^T = Q^T dS.
__global__ __launch_bounds__(256) void tf_attn_bwd_dkdv(TfAttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sq[64 * 64];
  __shared__ __attribute__((aligned(16))) uint16_t sdo[64 * 64];
  __shared__ float sl[64], sd[64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4;
  const int nb = (a.T + 63) / 64;
  const int kb = (int)blockIdx.x;  // the first key blocks see the most query blocks
  const int h = blockIdx.y, b = blockIdx.z;
  const int k0 = kb * 64;
  const int key = k0 + 16 * wave + (lane & 15);
  const int64_t base = (int64_t)b * a.T;
  const int64_t colq = (int64_t)h * 64, colk = a.d + colq, colv = 2 * (int64_t)a.d + colq;
  u32x4_t kf[2], vf[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    kf[s] = vf[s] = u32x4_t{0u, 0u, 0u, 0u};
    if (key < a.T) {
      kf[s] = *reinterpret_cast<const u32x4_t*>(a.qkv + (base + key) * a.ldqkv + colk + 32 * s + 8 * g);
      vf[s] = *reinterpret_cast<const u32x4_t*>(a.qkv + (base + key) * a.ldqkv + colv + 32 * s + 8 * g);
    }
  }
  const float sc = a.scale * kLog2e;
  const float* lse = a.lse + ((int64_t)b * a.H + h) * a.T;
  const float* dsum = a.dsum + ((int64_t)b * a.H + h) * a.T;
  f32x4_t dvt[4], dkt[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) dvt[dt] = dkt[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const uint16_t* qbase = a.qkv + base * a.ldqkv;
  const uint16_t* dobase = a.dout + base * a.lddo;
  Stage2 nq = load64(qbase, a.ldqkv, kb * 64, a.T, colq, tid), nd = load64(dobase, a.lddo, kb * 64, a.T, colq, tid);
  float nl = 0.f, ns = 0.f;
  if (tid < 64 && kb * 64 + tid < a.T) {
    nl = lse[kb * 64 + tid] * kLog2e;
    ns = dsum[kb * 64 + tid];
  }
  for (int qb = kb; qb < nb; ++qb) {
    const int q0 = qb * 64;
    __syncthreads();
    store64(sq, nq, tid);
    store64(sdo, nd, tid);
    if (tid < 64) {
      sl[tid] = nl;
      sd[tid] = ns;
    }
    __syncthreads();
    if (qb + 1 < nb) {  // next block's loads in flight during this block's compute
      nq = load64(qbase, a.ldqkv, q0 + 64, a.T, colq, tid);
      nd = load64(dobase, a.lddo, q0 + 64, a.T, colq, tid);
      nl = ns = 0.f;
      if (tid < 64 && q0 + 64 + tid < a.T) {
        nl = lse[q0 + 64 + tid] * kLog2e;
        ns = dsum[q0 + 64 + tid];
      }
    }
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      f32x4_t s4[2], p4[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        s4[t] = p4[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int qr = 32 * st + prow(lane, t);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          s4[t] = mfma(row_chunk(sq, qr, 4 * s + g), kf[s], s4[t]);
          p4[t] = mfma(row_chunk(sdo, qr, 4 * s + g), vf[s], p4[t]);
        }
      }
      float p[8], ds[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int ql = 32 * st + 8 * g + 4 * t + q;  // local query row
          const int qrow = q0 + ql;
          const bool ok = key <= qrow && qrow < a.T && key < a.T;
          const float pv = ok ? __builtin_amdgcn_exp2f(s4[t][q] * sc - sl[ql]) : 0.f;
          p[4 * t + q] = pv;
          ds[4 * t + q] = pv * (p4[t][q] - sd[ql]);
        }
      const u32x4_t pf = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
      const u32x4_t dsf = {pack2(ds[0], ds[1]), pack2(ds[2], ds[3]), pack2(ds[4], ds[5]), pack2(ds[6], ds[7])};
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        dvt[dt] = mfma(col_frag(sdo, 32 * st, 16 * dt, lane), pf, dvt[dt]);   // dV^T += dO^T P
        dkt[dt] = mfma(col_frag(sq, 32 * st, 16 * dt, lane), dsf, dkt[dt]);   // dK^T += Q^T dS
      }
    }
  }
  if (key < a.T) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      uint2 w;
      w.x = pack2(dkt[dt][0] * a.scale, dkt[dt][1] * a.scale);
      w.y = pack2(dkt[dt][2] * a.scale, dkt[dt][3] * a.scale);
      *reinterpret_cast<uint2*>(a.dqkv + (base + key) * a.lddqkv + colk + 16 * dt + 4 * g) = w;
      w.x = pack2(dvt[dt][0], dvt[dt][1]);
      w.y = pack2(dvt[dt][2], dvt[dt][3]);
      *reinterpret_cast<uint2*>(a.dqkv + (base + key) * a.lddqkv + colv + 16 * dt + 4 * g) = w;
    }
  }
}

// dQ of a query block: wave w owns query rows q0 + 16 w + (l & 15); for every
// key block at or before it, S^T and dP^T as in the forward, then
// dQ^T += K^T dS^T.
__global__ __launch_bounds__(256) void tf_attn_bwd_dq(TfAttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sk[64 * 64];
  __shared__ __attribute__((aligned(16))) uint16_t sv[64 * 64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4;
  const int nqb = (a.T + 63) / 64;
  const int qb = nqb - 1 - (int)blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int q0 = qb * 64;
  const int qrow = q0 + 16 * wave + (lane & 15);
  const int64_t base = (int64_t)b * a.T;
  const int64_t colq = (int64_t)h * 64, colk = a.d + colq, colv = 2 * (int64_t)a.d + colq;
  u32x4_t qf[2], df[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    qf[s] = df[s] = u32x4_t{0u, 0u, 0u, 0u};
    if (qrow < a.T) {
      qf[s] = *reinterpret_cast<const u32x4_t*>(a.qkv + (base + qrow) * a.ldqkv + colq + 32 * s + 8 * g);
      df[s] = *reinterpret_cast<const u32x4_t*>(a.dout + (base + qrow) * a.lddo + colq + 32 * s + 8 * g);
    }
  }
  const float sc = a.scale * kLog2e;
  const int64_t hrow = ((int64_t)b * a.H + h) * a.T;
  const float lq = qrow < a.T ? a.lse[hrow + qrow] * kLog2e : 0.f;
  const float dq = qrow < a.T ? a.dsum[hrow + qrow] : 0.f;
  f32x4_t acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const uint16_t* kvbase = a.qkv + base * a.ldqkv;
  Stage2 nk = load64(kvbase, a.ldqkv, 0, a.T, colk, tid), nv = load64(kvbase, a.ldqkv, 0, a.T, colv, tid);
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * 64;
    __syncthreads();
    store64(sk, nk, tid);
    store64(sv, nv, tid);
    __syncthreads();
    if (kb < qb) {
      nk = load64(kvbase, a.ldqkv, k0 + 64, a.T, colk, tid);
      nv = load64(kvbase, a.ldqkv, k0 + 64, a.T, colv, tid);
    }
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      f32x4_t s4[2], p4[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        s4[t] = p4[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int kr = 32 * st + prow(lane, t);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          s4[t] = mfma(row_chunk(sk, kr, 4 * s + g), qf[s], s4[t]);
          p4[t] = mfma(row_chunk(sv, kr, 4 * s + g), df[s], p4[t]);
        }
      }
      float ds[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int key = k0 + 32 * st + 8 * g + 4 * t + q;
          const bool ok = key <= qrow && key < a.T && qrow < a.T;
          const float pv = ok ? __builtin_amdgcn_exp2f(s4[t][q] * sc - lq) : 0.f;
          ds[4 * t + q] = pv * (p4[t][q] - dq);
        }
      const u32x4_t dsf = {pack2(ds[0], ds[1]), pack2(ds[2], ds[3]), pack2(ds[4], ds[5]), pack2(ds[6], ds[7])};
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) acc[dt] = mfma(col_frag(sk, 32 * st, 16 * dt, lane), dsf, acc[dt]);
    }
  }
  if (qrow < a.T) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      uint2 w;
      w.x = pack2(acc[dt][0] * a.scale, acc[dt][1] * a.scale);
      w.y = pack2(acc[dt][2] * a.scale, acc[dt][3] * a.scale);
      *reinterpret_cast<uint2*>(a.dqkv + (base + qrow) * a.lddqkv + colq + 16 * dt + 4 * g) = w;
    }
  }
}

// ---------------------------------------------------------------------------
// vocabulary head: softmax normaliser, loss and gradient scale per row
// ---------------------------------------------------------------------------
// Range of S_n (the sum of a row's exponentials relative to the target logit)
// the fast path accepts: S_n >= e^0 up to rounding whenever the target is
// valid, and S_n <= 2^60 keeps rowscale and hns far from underflow.
constexpr float kHeadLo = 0x1p-60f, kHeadHi = 0x1p60f;

// rowscale, the target entry of the gradient (pt: its stored exponential)
// and hns = rowscale hn of row n, by the lanes of one wave
__device__ __forceinline__ void head_finish(const TfHeadArgs& a, int64_t n, float se, int tg, float pt, int lane) {
  const float s = a.scale / se;
  if (lane == 0) {
    a.rowscale[n] = s;
    if (tg >= 0) a.e[n * a.lde + tg] = tobf(pt - se);
  }
  for (int c = lane; c < a.d / 8; c += 64) {
    const u32x4_t h = *reinterpret_cast<const u32x4_t*>(a.hn + n * a.ldhn + c * 8);
    u32x4_t o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = pack2(lo16(h[k]) * s, hi16(h[k]) * s);
    *reinterpret_cast<u32x4_t*>(a.hns + n * a.ldhns + c * 8) = o;
  }
}

__global__ __launch_bounds__(256) void tf_head_norm(TfHeadArgs a) {
  __shared__ float sloss[4];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + wave;
  float loss = 0.f;
  if (n < a.N) {
    const float* st = a.lstat + n * a.ldlstat;
    float se = 0.f;
    for (int t = lane; t < a.ntiles; t += 64) se += st[t];
    se = wsum(se);
    const int tg = a.target[n];
    if (se >= kHeadLo && se <= kHeadHi) {  // false for NaN
      loss = tg >= 0 ? __logf(se) : 0.f;
      const float pt = tg >= 0 ? bf(a.e[n * a.lde + tg]) : 0.f;
      head_finish(a, n, se, tg, pt, lane);
    } else if (lane == 0) {
      a.flag[n] = 1;
    }
    if (lane == 0) a.rowloss[n] = loss;
  }
  if (lane == 0) sloss[wave] = loss;
  __syncthreads();
  if (threadIdx.x == 0) a.ploss[blockIdx.x] = (sloss[0] + sloss[1]) + (sloss[2] + sloss[3]);
}

// logit of vocabulary row v from the head input held in LDS (fp32)
__device__ __forceinline__ float head_logit(const TfHeadArgs& a, const float* h, int v) {
  const uint16_t* w = a.w + (int64_t)v * a.ldw;
  float x = 0.f;
  for (int c = 0; c < a.d; c += 8) {
    const u32x4_t q = *reinterpret_cast<const u32x4_t*>(w + c);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x = fmaf(h[c + 2 * k], lo16(q[k]), x);
      x = fmaf(h[c + 2 * k + 1], hi16(q[k]), x);
    }
  }
  return x;
}

// Flagged rows of a group of four: the row's logits recomputed (one thread
// per vocabulary row, fp32 dot products), their exact maximum as the
// reference, then the exponentials, their sum and the same outputs as the
// fast path.  Sums in a fixed order (per thread over its rows, a wave
// butterfly, then the four waves).
constexpr int kHeadMaxD = 4096;
__global__ __launch_bounds__(256) void tf_head_fix(TfHeadArgs a) {
  __shared__ int fl[4];
  __shared__ float hrow[kHeadMaxD];
  __shared__ float red[3][4];
  __shared__ float spt;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t n0 = (int64_t)blockIdx.x * 4;
  if (tid < 4) fl[tid] = n0 + tid < a.N ? a.flag[n0 + tid] : 0;
  __syncthreads();
  if (!(fl[0] | fl[1] | fl[2] | fl[3])) return;
  for (int j = 0; j < 4; ++j) {
    if (!fl[j]) continue;
    const int64_t n = n0 + j;
    const int tg = a.target[n];
    for (int c = tid; c < a.d; c += 256) hrow[c] = bf(a.hn[n * a.ldhn + c]);
    if (tid == 0) spt = 0.f;
    __syncthreads();
    float mx = -INFINITY;
    for (int v = tid; v < a.V; v += 256) mx = fmaxf(mx, head_logit(a, hrow, v));
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    float se = 0.f, xt = 0.f;
    for (int v = tid; v < a.V; v += 256) {
      const float x = head_logit(a, hrow, v);
      const uint16_t p = tobf(__expf(x - mx));
      a.e[n * a.lde + v] = p;
      se += bf(p);
      if (v == tg) {
        xt = x;
        spt = bf(p);
      }
    }
    se = wsum(se);
    xt = wsum(xt);  // one thread holds the target logit, the others zero
    if (lane == 0) {
      red[1][wave] = se;
      red[2][wave] = xt;
    }
    __syncthreads();
    se = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    xt = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
    if (wave == 0) head_finish(a, n, se, tg, spt, lane);
    if (tid == 0) {
      a.rowloss[n] = tg >= 0 ? mx + __logf(se) - xt : 0.f;
      a.flag[n] = 0;
    }
    __syncthreads();
  }
  if (tid == 0) {
    float l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) l[q] = n0 + q < a.N ? a.rowloss[n0 + q] : 0.f;
    a.ploss[blockIdx.x] = (l[0] + l[1]) + (l[2] + l[3]);
  }
}

// ---------------------------------------------------------------------------
// embedding gradient
// ---------------------------------------------------------------------------
// counts per token (integer counters: the result does not depend on order;
// they start at zero and tf_emb_rows clears them after use)
__global__ __launch_bounds__(256) void tf_emb_count(TfEmbGradArgs a) {
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n < a.N) {
    const int32_t t = a.input[n];
    if (t >= 0) atomicAdd(&a.count[t], 1);
  }
}

// exclusive prefix sum of the counts (one workgroup of 1024 threads), and
// the fill counters back to zero
__global__ __launch_bounds__(1024) void tf_emb_scan(TfEmbGradArgs a) {
  __shared__ int part[1024];
  const int tid = threadIdx.x;
  const int per = (a.V + 1023) / 1024;
  const int lo = tid * per, hi = min(a.V, lo + per);
  int s = 0;
  for (int v = lo; v < hi; ++v) s += a.count[v];
  part[tid] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {  // inclusive Hillis-Steele scan
    const int x = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  int run = part[tid] - s;
  for (int v = lo; v < hi; ++v) {
    a.start[v] = run;
    run += a.count[v];
    a.fill[v] = 0;
  }
}

// every position into its token's bucket (order inside a bucket arbitrary)
__global__ __launch_bounds__(256) void tf_emb_scatter(TfEmbGradArgs a) {
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n < a.N) {
    const int32_t t = a.input[n];
    if (t >= 0) a.bucket[a.start[t] + atomicAdd(&a.fill[t], 1)] = (int32_t)n;
  }
}

// one wave per vocabulary row: the bucket's positions are visited in
// increasing order (each step takes the smallest position above the last
// one, a wave-wide minimum) and their gradient rows summed in that order;
// rows of absent tokens are zero.  The row's counter is cleared for the next
// step.  At most 4096 columns (16 float4 per lane).
constexpr int kEmbVec = 16;
__global__ __launch_bounds__(256) void tf_emb_rows(TfEmbGradArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t v = (int64_t)blockIdx.x * 4 + wave;
  if (v >= a.V) return;
  const int s0 = a.start[v], c = a.count[v];
  const int32_t mine = lane < c ? a.bucket[s0 + lane] : INT32_MAX;
  float4 acc[kEmbVec];
#pragma unroll
  for (int i = 0; i < kEmbVec; ++i) acc[i] = make_float4(0.f, 0.f, 0.f, 0.f);
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
    const float* row = a.dx + (int64_t)cand * a.lddx;
#pragma unroll
    for (int i = 0; i < kEmbVec; ++i) {
      const int cc = lane + 64 * i;
      if (cc < a.d / 4) {
        const float4 x = *reinterpret_cast<const float4*>(row + cc * 4);
        acc[i].x += x.x;
        acc[i].y += x.y;
        acc[i].z += x.z;
        acc[i].w += x.w;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < kEmbVec; ++i) {
    const int cc = lane + 64 * i;
    if (cc < a.d / 4) *reinterpret_cast<float4*>(a.grad + v * a.ldgrad + cc * 4) = acc[i];
  }
  if (lane == 0) a.count[v] = 0;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_tf_embed(const TfEmbedArgs& a, hipStream_t s, const LaunchEv& ev) {
  const int64_t n = (int64_t)a.B * a.T;
  ERASE_TF_LAUNCH(tf_embed, dim3((unsigned)((n + 3) / 4)), dim3(256), s, ev, a);
  return hipGetLastError();
}

hipError_t launch_tf_rms(int backward, const TfRmsArgs& a, hipStream_t s, const LaunchEv& ev) {
  if (a.d % 8 || a.d > 64 * 8 * kRmsChunks) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.N + 3) / 4));
  if (backward)
    ERASE_TF_LAUNCH(tf_rms_bwd, grid, dim3(256), s, ev, a);
  else
    ERASE_TF_LAUNCH(tf_rms_fwd, grid, dim3(256), s, ev, a);
  return hipGetLastError();
}

hipError_t launch_tf_attn(int part, const TfAttnArgs& a, hipStream_t s, const LaunchEv& ev) {
  const dim3 grid((unsigned)((a.T + 63) / 64), (unsigned)a.H, (unsigned)a.B);
  switch (part) {
    case 0: ERASE_TF_LAUNCH(tf_attn_fwd, grid, dim3(256), s, ev, a); break;
    case 1: {
      const int64_t rows = (int64_t)a.B * a.T * a.H;
      ERASE_TF_LAUNCH(tf_attn_bwd_pre, dim3((unsigned)((rows + 31) / 32)), dim3(256), s, ev, a);
      break;
    }
    case 2: ERASE_TF_LAUNCH(tf_attn_bwd_dkdv, grid, dim3(256), s, ev, a); break;
    case 3: ERASE_TF_LAUNCH(tf_attn_bwd_dq, grid, dim3(256), s, ev, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_tf_head(int part, const TfHeadArgs& a, hipStream_t s, const LaunchEv& ev) {
  if (a.d % 8 || a.d > kHeadMaxD || a.N < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.N + 3) / 4));
  if (part == 0)
    ERASE_TF_LAUNCH(tf_head_norm, grid, dim3(256), s, ev, a);
  else
    ERASE_TF_LAUNCH(tf_head_fix, grid, dim3(256), s, ev, a);
  return hipGetLastError();
}

hipError_t launch_tf_emb_grad(const TfEmbGradArgs& a, hipStream_t s) {
  if (a.d % 4 || a.d > 4 * 64 * kEmbVec) return hipErrorInvalidValue;
  const dim3 gn((unsigned)((a.N + 255) / 256));
  hipLaunchKernelGGL(tf_emb_count, gn, dim3(256), 0, s, a);
  hipLaunchKernelGGL(tf_emb_scan, dim3(1), dim3(1024), 0, s, a);
  hipLaunchKernelGGL(tf_emb_scatter, gn, dim3(256), 0, s, a);
  hipLaunchKernelGGL(tf_emb_rows, dim3((unsigned)((a.V + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace erase
