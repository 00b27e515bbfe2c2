// C-ABI entry points, host validation, workspace layout and the two-stream
// dispatcher of the ERASE detached-block step.
//
// Schedules (paper, Section 2.2): conventional training runs the backward
// after the whole forward; ERASE launches block b's backward on a second
// stream as soon as its forward and local loss are done, with events
// enforcing the remaining dependencies, so it overlaps block b+1's forward.
// HIP graphs fix the launch order and remove per-launch host cost (the
// paper's CUDA-Graph variant).  A worker host thread can enqueue the backward
// streams' work while the calling thread enqueues the next forward (the
// paper's non-blocking dispatch).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <deque>
#include <functional>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "erase.h"
#include "internal.h"

namespace {

using namespace erase;

constexpr int kMaxBlocks = 64;
constexpr int kMaxLayers = 16;
constexpr int64_t kMaxDim = 65536;
constexpr int64_t kMaxBatch = int64_t(1) << 24;
constexpr size_t kAlign = 256;
constexpr int kMaxGraphs = 32;
constexpr int kMaxBwdStreams = 8;

int64_t roundup(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------
// validation (host only, no HIP call)
// ---------------------------------------------------------------------------
erase_status validate(const erase_config* c, std::string* err) {
  auto fail = [&](erase_status s, const char* msg) {
    if (err) *err = msg;
    return s;
  };
  if (!c) return fail(ERASE_ERR_INVALID_ARG, "config is NULL");
  if (c->dtype != ERASE_F32 && c->dtype != ERASE_BF16) return fail(ERASE_ERR_INVALID_ARG, "dtype must be F32 or BF16");
  if (c->n_blocks < 1 || c->n_blocks > kMaxBlocks) return fail(ERASE_ERR_SHAPE, "n_blocks must be in [1, 64]");
  if (!c->blocks) return fail(ERASE_ERR_INVALID_ARG, "blocks is NULL");
  if (c->batch < 1 || c->batch > kMaxBatch) return fail(ERASE_ERR_SHAPE, "batch must be in [1, 2^24]");
  if (c->in_dim < 1 || c->in_dim > kMaxDim) return fail(ERASE_ERR_SHAPE, "in_dim must be in [1, 65536]");
  const int esz = c->dtype == ERASE_BF16 ? 2 : 4;
  if (c->x_ld < c->in_dim || (int64_t(c->x_ld) * esz) % 16 != 0)
    return fail(ERASE_ERR_SHAPE, "x_ld must be >= in_dim and a multiple of 16 bytes");
  if (c->x_in_place != 0 && c->x_in_place != 1) return fail(ERASE_ERR_INVALID_ARG, "x_in_place must be 0 or 1");
  if (c->x_in_place && (c->x_ld % 128 != 0 || c->batch % 128 != 0))
    return fail(ERASE_ERR_SHAPE, "x read in place: x_ld and batch must be multiples of 128");
  if (!(std::isfinite(c->lr) && c->lr >= 0.f)) return fail(ERASE_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (!(c->beta1 >= 0.f && c->beta1 < 1.f && c->beta2 >= 0.f && c->beta2 < 1.f))
    return fail(ERASE_ERR_INVALID_ARG, "betas must be in [0, 1)");
  if (!(std::isfinite(c->eps) && c->eps >= 0.f)) return fail(ERASE_ERR_INVALID_ARG, "eps must be finite and >= 0");
  int prev_out = -1;
  for (int b = 0; b < c->n_blocks; ++b) {
    const erase_block_spec& B = c->blocks[b];
    if (B.input_src != ERASE_IN_X && B.input_src != ERASE_IN_PREV)
      return fail(ERASE_ERR_INVALID_ARG, "input_src must be IN_X or IN_PREV");
    if (b == 0 && B.input_src != ERASE_IN_X) return fail(ERASE_ERR_INVALID_ARG, "block 0 must read x");
    if (B.n_layers < 1 || B.n_layers > kMaxLayers) return fail(ERASE_ERR_SHAPE, "n_layers must be in [1, 16]");
    if (!B.layers) return fail(ERASE_ERR_INVALID_ARG, "layers is NULL");
    if (B.loss != ERASE_LOSS_BCE) return fail(ERASE_ERR_UNSUPPORTED, "only the sigmoid-BCE local loss is implemented");
    if (!std::isfinite(B.lambda)) return fail(ERASE_ERR_INVALID_ARG, "lambda must be finite");
    const int width = B.input_src == ERASE_IN_X ? c->in_dim : prev_out;
    int cur = width;
    bool seen_linear = false;
    for (int l = 0; l < B.n_layers; ++l) {
      const erase_layer_spec& L = B.layers[l];
      if (L.kind != ERASE_LAYER_LINEAR_RELU && L.kind != ERASE_LAYER_CROSS)
        return fail(ERASE_ERR_INVALID_ARG, "layer kind must be LINEAR_RELU or CROSS");
      if (L.in_dim < 1 || L.in_dim > kMaxDim || L.out_dim < 1 || L.out_dim > kMaxDim)
        return fail(ERASE_ERR_SHAPE, "layer dims must be in [1, 65536]");
      if (L.in_dim != cur) return fail(ERASE_ERR_SHAPE, "layer in_dim does not match the width feeding it");
      if (int64_t(L.in_dim) * L.out_dim > (int64_t(1) << 31) - 1)
        return fail(ERASE_ERR_SHAPE, "layer weight has more than 2^31-1 elements");
      if (L.kind == ERASE_LAYER_CROSS) {
        if (seen_linear) return fail(ERASE_ERR_UNSUPPORTED, "cross layers must precede linear layers");
        if (L.out_dim != L.in_dim || L.in_dim != width)
          return fail(ERASE_ERR_SHAPE, "a cross layer keeps the block input width");
      } else {
        seen_linear = true;
      }
      cur = L.out_dim;
    }
    if (B.layers[B.n_layers - 1].kind != ERASE_LAYER_LINEAR_RELU)
      return fail(ERASE_ERR_UNSUPPORTED, "the last layer of a block must be LINEAR_RELU");
    if (cur > HEAD_MAX_N) return fail(ERASE_ERR_UNSUPPORTED, "the head input width must be <= 2048");
    prev_out = cur;
  }
  return ERASE_OK;
}

// ---------------------------------------------------------------------------
// plan: every buffer of the workspace and every launch's shape
// ---------------------------------------------------------------------------
struct GemmPlan {
  int bm = 64, bn = 64, split = 1, kps = 0;
  int group = 0;    // XCD-aware tile order (xcd_group), set once the plan is final
  int kgroups = 1;  // k-groups of four waves per workgroup
};

struct LayerRT {
  int kind = 0, K = 0, N = 0;
  int64_t offW = 0, offb = 0;
  void* wsh = nullptr; int64_t ldwsh = 0;
  void* wsht = nullptr; int64_t ldwsht = 0;
  void* y = nullptr; int64_t ldy = 0;      // activation [Mr][ldy]
  bool needy = true;                        // y is read later (not a fused head's unchained output)
  void* dmn = nullptr; int64_t lddmn = 0;  // activation gradient [Mr][lddmn]
  void* g = nullptr; int64_t ldg = 0;
  float* part = nullptr; int64_t ldp = 0, pstride = 0;
  float* bpart = nullptr;
  GemmPlan fwd, wgrad, dgrad;
  bool grouped = false;  // input- and weight-gradient GEMMs share one launch
  // Adam of the weight matrix fused into its (standalone, unsplit, two
  // k-group) weight-gradient launch
  bool fused_adam = false;
};

struct BlockRT {
  int input_src = 0;
  float lam = 1.f;
  int L = 0;
  LayerRT layer[kMaxLayers];
  int64_t nparam = 0, off_w = 0, off_c = 0;
  bool send = false;  // undetached schedule: the input gradient goes back to the previous block
  int nhead = 0;      // head partial rows (M-tiles of the head)
  bool head_fused = false;  // head+loss in the last forward GEMM's epilogue
  float* pdw = nullptr;
  float* pdc = nullptr;
  float* ploss = nullptr;
  AdamSeg* segs_dev = nullptr;   // segments the Adam kernel updates
  AdamSeg* rsegs_dev = nullptr;  // every segment (GEMM-copy refresh)
  std::vector<AdamSeg> rsegs;
  int64_t rnchunks = 0;
  std::vector<AdamSeg> segs;
  int64_t nchunks = 0;
  erase_block_buffers buf{};
};

struct Plan {
  int bf16 = 1, esz = 2, M = 0;
  bool undet_ok = true;  // every chained block can send its input gradient back
  int64_t Mr = 0;   // allocated rows of row-major arrays: roundup(M, 128)
  int64_t* t = nullptr;
  int* status = nullptr;
  // zero-padded and feature-major copies of x, one pair per step parity so a
  // step's prologue never overwrites what the previous step's backward reads
  void* xp[2] = {nullptr, nullptr}; int64_t ldxp = 0;
  bool x_in_place = false;  // the GEMMs read the caller's (zero-padded) x; no copy

  std::vector<BlockRT> blk;
  size_t bytes = 0;
};

struct Carver {
  uintptr_t base;
  size_t off = kAlign;  // the first 256 bytes hold the step counter and status word
  void* take(size_t n) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    void* p = reinterpret_cast<void*>(base + off);
    off += std::max<size_t>(n, 1);
    return p;
  }
};

// Workgroup tile and split of one GEMM.  Enough workgroups to cover the 256
// CUs when the shape allows it, the largest tile that still does, and a
// split of the contraction only for weight gradients (whose outputs are few).
GemmPlan choose_gemm(int bf16, int64_t Mg, int64_t Ng, int64_t Kc, bool allow_split) {
  GemmPlan p;
  const int BK = bf16 ? 64 : 32;
  auto finish = [&](int bm, int bn, int split) {
    p.bm = bm;
    p.bn = bn;
    p.kps = (int)roundup(cdiv(std::max<int64_t>(Kc, 1), split), BK);
    p.split = (int)cdiv(std::max<int64_t>(Kc, 1), p.kps);
    return p;
  };
  if (!bf16) return finish(64, 64, 1);
  // At least `target` workgroups (1.5 per CU) so the launch covers the
  // chip; the largest tile that reaches it (fewer LDS bytes per MFMA).  A
  // long contraction (>= 1024) takes one 64x128 workgroup per CU over two
  // 64x64 ones (4096 x 512 x 1728: 14.7 vs 15.8 us).  Otherwise a short
  // contraction falls back to 64x64, split only for weight gradients (a
  // 128x64 split 4 of the 512 x 1677 weight gradient over 4096 rows is 1.5
  // us faster than 64x64 split 2, but its two extra partial slices cost
  // Adam 2.1 us more).
  const int64_t target = 384;
  auto wgs = [&](int bm, int bn) { return cdiv(Mg, bm) * cdiv(Ng, bn); };
  const int tiles[3][2] = {{128, 128}, {128, 64}, {64, 128}};
  for (int i = 0; i < 3; ++i)
    if (wgs(tiles[i][0], tiles[i][1]) >= target) return finish(tiles[i][0], tiles[i][1], 1);
  if (!allow_split && Kc >= 1024 && wgs(64, 128) >= 256) {
    // one workgroup per CU: two k-groups give each SIMD two waves
    p.kgroups = 2;
    return finish(64, 128, 1);
  }
  if (wgs(64, 64) >= target) return finish(64, 64, 1);
  // at most one 64x64 workgroup per CU: two k-groups give each SIMD two waves
  if (!allow_split && wgs(64, 64) <= 256) p.kgroups = 2;
  if (allow_split) {
    int s = 1;
    while (s < 16 && wgs(128, 128) * s < target && Kc / (s * 2) >= 2048) s *= 2;
    if (wgs(128, 128) * s >= target) return finish(128, 128, s);
    s = 1;
    while (s < 16 && wgs(64, 64) * s < target && Kc / (s * 2) >= 256) s *= 2;
    return finish(64, 64, s);
  }
  return finish(64, 64, 1);
}

size_t build_plan(const erase_config& c, uintptr_t base, Plan* P) {
  P->bf16 = c.dtype == ERASE_BF16;
  P->esz = P->bf16 ? 2 : 4;
  P->M = c.batch;
  const int esz = P->esz;
  const int64_t M = c.batch;
  P->Mr = roundup(M, 128);
  const int64_t Mr = P->Mr;
  Carver cv{base};
  P->t = reinterpret_cast<int64_t*>(base);
  P->status = reinterpret_cast<int*>(base + 8);
  bool any_x = false;
  for (int b = 0; b < c.n_blocks; ++b) any_x |= c.blocks[b].input_src == ERASE_IN_X;
  P->x_in_place = c.x_in_place != 0;
  if (any_x && !P->x_in_place) {
    // zero-padded copy of x, one per step parity; 128-column rows (the
    // weight gradient reads k-major tiles up to 128 columns wide)
    P->ldxp = roundup(c.in_dim, 128);
    for (int q = 0; q < 2; ++q) P->xp[q] = cv.take(size_t(Mr) * P->ldxp * esz);
  }
  P->blk.assign(c.n_blocks, BlockRT{});
  for (int b = 0; b < c.n_blocks; ++b) {
    const erase_block_spec& S = c.blocks[b];
    BlockRT& B = P->blk[b];
    B.input_src = S.input_src;
    B.lam = S.lambda;
    B.L = S.n_layers;
    const bool next_chained = b + 1 < c.n_blocks && c.blocks[b + 1].input_src == ERASE_IN_PREV;
    int64_t off = 0;
    for (int l = 0; l < B.L; ++l) {
      LayerRT& R = B.layer[l];
      R.kind = S.layers[l].kind;
      R.K = S.layers[l].in_dim;
      R.N = S.layers[l].out_dim;
      R.offW = off;
      off += int64_t(R.K) * R.N;
      R.offb = off;
      off += R.N;
      // Every GEMM operand is zero-padded: weight copies to rows of a
      // multiple of 128 (the largest tile) and a leading dimension of a
      // multiple of 64 (the k-step); activations and their gradients to
      // roundup(M, 128) rows of a multiple of 128 columns (the k-major
      // weight-gradient tiles).
      const int64_t ldK = roundup(R.K, 64), ldN = roundup(R.N, 64);
      const int64_t Kr = roundup(R.K, 128), Nr = roundup(R.N, 128);
      R.ldwsh = ldK;
      R.wsh = cv.take(size_t(Nr) * ldK * esz);
      // the input gradient of a layer: every layer but a block's first, and
      // (undetached schedule) the first layer of a block reading the
      // previous block's output
      const bool dgrad = l >= 1 || S.input_src == ERASE_IN_PREV;
      if (dgrad) {
        R.ldwsht = ldN;
        R.wsht = cv.take(size_t(Kr) * ldN * esz);
      }
      R.ldy = Nr;
      R.y = cv.take(size_t(Mr) * Nr * esz);
      R.needy = l + 1 < B.L || next_chained;
      R.lddmn = Nr;
      R.dmn = cv.take(size_t(Mr) * Nr * esz);
      if (R.kind == ERASE_LAYER_CROSS && l >= 1) {
        R.ldg = Nr;
        R.g = cv.take(size_t(Mr) * Nr * esz);
      }
      // launch shapes (contraction lengths padded to the k-step)
      const int BK = P->bf16 ? 64 : 32;
      R.fwd = choose_gemm(P->bf16, M, R.N, roundup(R.K, BK), false);
      R.wgrad = choose_gemm(P->bf16, R.N, R.K, roundup(M, BK), true);
      if (l == 0 && dgrad) {
        R.dgrad = choose_gemm(P->bf16, M, R.K, roundup(R.N, BK), false);
        R.dgrad.group = xcd_group((int)cdiv(M, R.dgrad.bm), (int)cdiv(R.K, R.dgrad.bn), 1, R.dgrad.bm, R.dgrad.bn);
      }
      if (l >= 1) {
        R.dgrad = choose_gemm(P->bf16, M, R.K, roundup(R.N, BK), false);
        // one launch for both backward GEMMs when they can share a tile
        if (R.dgrad.bm != R.wgrad.bm || R.dgrad.bn != R.wgrad.bn) {
          GemmPlan d64 = choose_gemm(P->bf16, 1, 1, roundup(R.N, BK), false);  // 64x64, split 1
          d64.kgroups = 1;  // the grouped launch runs 256-thread workgroups at 64x64
          GemmPlan w64 = d64;
          const int64_t w = cdiv(R.N, 64) * cdiv(R.K, 64);
          int sp = 1;
          while (sp < 16 && w * sp < 384 && roundup(M, BK) / (sp * 2) >= 256) sp *= 2;
          w64.kps = (int)roundup(cdiv(roundup(M, BK), sp), BK);
          w64.split = (int)cdiv(roundup(M, BK), w64.kps);
          R.dgrad = d64;
          R.wgrad = w64;
        }
        R.grouped = (R.dgrad.bm == 64 && R.dgrad.bn == 64) || (R.dgrad.bm == 128 && R.dgrad.bn == 128);
        if (R.grouped && R.wgrad.split > 1) {
          // the input-gradient tiles of the same launch fill the chip: the
          // weight gradient keeps slices of >= 512 batch rows, so Adam reads
          // fewer fp32 partial slices.  CTR layers 2 and 3, A/B on one MI355X of
          // 4, 8 and 16 slices: the launch 10.9, 9.2, 9.2 us; SERIAL 9.36M,
          // 9.78M, 9.51M samples/s; PIPELINE+worker 12.85M, 12.94M, 12.38M
          // (16 slices: the first layer's launch, whose extra workgroups run
          // the other layers' Adam, 22.1 -> 23.5 us)
          const int64_t Kc = roundup(M, BK);
          int sp = R.wgrad.split;
          while (sp > 1 && Kc / sp < 512) sp /= 2;
          R.wgrad.kps = (int)roundup(cdiv(Kc, sp), BK);
          R.wgrad.split = (int)cdiv(Kc, R.wgrad.kps);
        }
        R.dgrad.group = xcd_group((int)cdiv(M, R.dgrad.bm), (int)cdiv(R.K, R.dgrad.bn), 1, R.dgrad.bm, R.dgrad.bn);
      }
      R.fwd.group = xcd_group((int)cdiv(M, R.fwd.bm), (int)cdiv(R.N, R.fwd.bn), 1, R.fwd.bm, R.fwd.bn);
      R.wgrad.group = xcd_group((int)cdiv(R.N, R.wgrad.bm), (int)cdiv(R.K, R.wgrad.bn), R.wgrad.split, R.wgrad.bm,
                                R.wgrad.bn);
      R.ldp = ldK;
      R.pstride = int64_t(R.N) * ldK;
      // A block's first layer has a weight-gradient launch of its own: its
      // workgroups hold whole 64x64 tiles of the gradient (two k-groups of
      // four waves over the whole batch, no split), so the layer's Adam runs
      // in that launch's epilogue and no partial slice goes to memory.  Not
      // when the transposed GEMM copy is needed (the undetached schedule's
      // input gradient), which only the Adam kernel writes.
      if (l == 0 && !dgrad) {
        R.fused_adam = true;
        R.wgrad.bm = R.wgrad.bn = 64;
        R.wgrad.split = 1;
        R.wgrad.kps = (int)roundup(M, BK);
        R.wgrad.kgroups = 2;
        R.wgrad.group = xcd_group((int)cdiv(R.N, 64), (int)cdiv(R.K, 64), 1, 64, 64);
      }
      R.part = static_cast<float*>(cv.take(size_t(R.wgrad.split) * R.pstride * 4));
      R.bpart = static_cast<float*>(cv.take(size_t(R.wgrad.split) * R.N * 4));
    }
    if (S.input_src == ERASE_IN_PREV) {
      // the gradient at this block's input reaches the previous block's
      // output through a linear+ReLU first layer into a linear+ReLU last layer
      const erase_block_spec& Sp = c.blocks[b - 1];
      B.send = S.layers[0].kind == ERASE_LAYER_LINEAR_RELU &&
               Sp.layers[Sp.n_layers - 1].kind == ERASE_LAYER_LINEAR_RELU;
      P->undet_ok = P->undet_ok && B.send;
    }
    const int NL = B.layer[B.L - 1].N;
    B.off_w = off;
    off += NL;
    B.off_c = off;
    off += 1;
    B.nparam = off;
    // Head+loss fused into the last forward GEMM when one tile spans the
    // whole width: 16 x 128 (bf16, a kernel of its own) or 64 x 64 (fp32,
    // the GEMM core) workgroups over M.  The layer is a few k-steps and the
    // head a chain of short dependent steps per workgroup, so shorter tiles
    // (more workgroups) win: 64-row GEMM-core tiles 12.1 us, 32-row 9.0 us
    // on the 4096 x 128 CTR layer.
    LayerRT& RL = B.layer[B.L - 1];
    B.head_fused = RL.kind == ERASE_LAYER_LINEAR_RELU && NL <= (P->bf16 ? 128 : 64);
    if (B.head_fused) {
      RL.fwd.bm = P->bf16 ? 16 : 64;
      RL.fwd.bn = P->bf16 ? 128 : 64;
      RL.fwd.kgroups = 1;
      RL.fwd.group = xcd_group((int)cdiv(M, RL.fwd.bm), 1, 1, RL.fwd.bm, RL.fwd.bn);
      B.nhead = (int)cdiv(M, RL.fwd.bm);
    } else {
      B.nhead = (int)cdiv(M, head_rows(NL, esz));
    }
    B.pdw = static_cast<float*>(cv.take(size_t(B.nhead) * NL * 4));
    B.pdc = static_cast<float*>(cv.take(size_t(B.nhead) * 4));
    B.ploss = static_cast<float*>(cv.take(size_t(B.nhead) * 4));
    const int nseg = 2 * B.L + 2;
    B.segs_dev = static_cast<AdamSeg*>(cv.take(sizeof(AdamSeg) * nseg));
    B.rsegs_dev = static_cast<AdamSeg*>(cv.take(sizeof(AdamSeg) * nseg));
  }
  P->bytes = cv.off;
  return cv.off;
}

// Adam segment tables (host copies; pointers into caller buffers/workspace).
void build_segments(Plan* P, const erase_block_buffers* bufs) {
  for (size_t b = 0; b < P->blk.size(); ++b) {
    BlockRT& B = P->blk[b];
    B.buf = bufs[b];
    B.segs.clear();
    B.rsegs.clear();
    int64_t chunk = 0, rchunk = 0;
    bool fused = false;  // the segment being added is updated by its weight-gradient launch
    auto add = [&](int64_t off, int rows, int cols, const float* part, int64_t pstride, int ldpart, int nsplit,
                    void* sh, int64_t ldsh, void* sht, int64_t ldsht) {
      AdamSeg s{};
      s.p = B.buf.param + off;
      s.m = B.buf.m + off;
      s.v = B.buf.v + off;
      s.g = B.buf.grad ? B.buf.grad + off : nullptr;
      s.part = part;
      s.pstride = pstride;
      s.rows = rows;
      s.cols = cols;
      s.ldpart = ldpart;
      s.nsplit = nsplit;
      s.sh = sh;
      s.ldsh = ldsh;
      s.sht = sht;
      s.ldsht = ldsht;
      s.tcols = (int)cdiv(cols, ADAM_TC);
      s.chunk0 = rchunk;
      rchunk += cdiv(rows, ADAM_TR) * s.tcols;
      B.rsegs.push_back(s);
      if (fused) return;
      s.chunk0 = chunk;
      chunk += cdiv(rows, ADAM_TR) * s.tcols;
      B.segs.push_back(s);
    };
    for (int l = 0; l < B.L; ++l) {
      LayerRT& R = B.layer[l];
      // a fused layer's weight and bias are updated by its weight-gradient launch
      fused = R.fused_adam;
      add(R.offW, R.N, R.K, R.part, R.pstride, (int)R.ldp, R.wgrad.split, R.wsh, R.ldwsh, R.wsht, R.ldwsht);
      add(R.offb, 1, R.N, R.bpart, R.N, R.N, R.wgrad.split, nullptr, 0, nullptr, 0);
      fused = false;
    }
    const int NL = B.layer[B.L - 1].N;
    add(B.off_w, 1, NL, B.pdw, NL, NL, B.nhead, nullptr, 0, nullptr, 0);
    add(B.off_c, 1, 1, B.pdc, 1, 1, B.nhead, nullptr, 0, nullptr, 0);
    B.nchunks = chunk;
    B.rnchunks = rchunk;
  }
}

// ---------------------------------------------------------------------------
// context
// ---------------------------------------------------------------------------
struct TimedLaunch {
  erase_kernel_time rec;
  hipEvent_t e0, e1;
};

struct GraphEntry {
  const void* x;
  const float* y;
  float* losses;
  int sched;
  int par;
  hipGraph_t graph;
  hipGraphExec_t exec;
};

// Error state of HIP calls made on a worker thread: hip_ok reports there
// instead of into the context, which only the calling thread writes.
struct ErrSink {
  erase_status st = ERASE_OK;
  std::string msg;
};
thread_local ErrSink* tl_sink = nullptr;

// One host thread running enqueue jobs in submission order.  Jobs are
// numbered from 1; wait(id) returns once jobs 1..id have finished.  After a
// failed job the remaining ones are skipped (counted as finished), and the
// first error is kept until take_error().
class Worker {
 public:
  explicit Worker(int device) : device_(device) { th_ = std::thread([this] { loop(); }); }
  ~Worker() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    th_.join();
  }
  uint64_t push(std::function<erase_status()> f) {
    std::lock_guard<std::mutex> lk(mu_);
    jobs_.push_back(std::move(f));
    const uint64_t id = ++pushed_;
    cv_.notify_all();
    return id;
  }
  void wait(uint64_t id) {
    std::unique_lock<std::mutex> lk(mu_);
    done_cv_.wait(lk, [&] { return done_ >= id; });
  }
  void drain() {
    std::unique_lock<std::mutex> lk(mu_);
    done_cv_.wait(lk, [&] { return done_ >= pushed_; });
  }
  bool take_error(ErrSink* out) {
    std::lock_guard<std::mutex> lk(mu_);
    if (err_.st == ERASE_OK) return false;
    *out = err_;
    err_ = ErrSink{};
    return true;
  }

 private:
  void loop() {
    (void)hipSetDevice(device_);
    for (;;) {
      std::function<erase_status()> f;
      bool skip;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return stop_ || !jobs_.empty(); });
        if (jobs_.empty()) return;  // stop requested and nothing left
        f = std::move(jobs_.front());
        jobs_.pop_front();
        skip = err_.st != ERASE_OK;
      }
      ErrSink local;
      erase_status st = ERASE_OK;
      if (!skip) {
        tl_sink = &local;
        st = f();
        tl_sink = nullptr;
      }
      {
        std::lock_guard<std::mutex> lk(mu_);
        if (st != ERASE_OK && err_.st == ERASE_OK) {
          err_.st = st;
          err_.msg = local.msg.empty() ? "backward enqueue failed on the worker thread" : local.msg;
        }
        ++done_;
      }
      done_cv_.notify_all();
    }
  }
  int device_;
  std::mutex mu_;
  std::condition_variable cv_, done_cv_;
  std::deque<std::function<erase_status()>> jobs_;
  uint64_t pushed_ = 0, done_ = 0;
  bool stop_ = false;
  ErrSink err_;
  std::thread th_;
};

struct Ctx {
  erase_config cfg{};
  std::vector<erase_block_spec> blocks;
  std::vector<std::vector<erase_layer_spec>> layers;
  Plan P;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t sf = nullptr;
  std::vector<hipStream_t> sbs;  // backward streams; block b uses sbs[b % size]
  int device = 0;
  std::vector<hipEvent_t> ef, eb;
  erase_status sticky = ERASE_OK;
  std::string err;
  std::vector<GraphEntry> graphs;
  bool timing = false;
  std::vector<hipEvent_t> tev;  // timing events pool
  hipEvent_t tstart = nullptr;
  hipEvent_t tnull0 = nullptr, tnull1 = nullptr;  // empty interval: event overhead
  std::vector<TimedLaunch> last;
  bool last_valid = false;
  int64_t hstep = 0;     // host copy of the step counter (steps enqueued)
  int par = 0;           // parity of the step being enqueued
  bool pending = false;  // a PIPELINE step left backward work unjoined
  // worker dispatch: the backward streams' launches are enqueued by
  // `worker` (created on first use); job_of[b] is the job that enqueued
  // block b's backward most recently
  bool use_worker = false;
  std::unique_ptr<Worker> worker;
  std::vector<uint64_t> job_of;
};

bool hip_ok(Ctx* c, hipError_t e, const char* what) {
  if (e == hipSuccess) return true;
  char buf[256];
  std::snprintf(buf, sizeof buf, "%s: %s", what, hipGetErrorString(e));
  if (tl_sink) {  // worker thread: reported when the calling thread joins it
    if (tl_sink->st == ERASE_OK) {
      tl_sink->st = ERASE_ERR_HIP;
      tl_sink->msg = buf;
    }
  } else if (c) {
    c->err = buf;
    c->sticky = ERASE_ERR_HIP;
  }
  return false;
}

// Wait for every job handed to the worker (if any) and move its first error
// into the context.  Every entry point that enqueues or reads stream work
// calls this first.
erase_status quiesce(Ctx* c) {
  if (!c->worker) return ERASE_OK;
  c->worker->drain();
  ErrSink e;
  if (c->worker->take_error(&e)) {
    c->err = e.msg;
    c->sticky = e.st;
    return e.st;
  }
  return ERASE_OK;
}

// Wait for worker job `id` (and those before it); its error, if any, goes
// into the context.
erase_status wait_job(Ctx* c, uint64_t id) {
  if (!c->worker || id == 0) return ERASE_OK;
  c->worker->wait(id);
  ErrSink e;
  if (c->worker->take_error(&e)) {
    c->err = e.msg;
    c->sticky = e.st;
    return e.st;
  }
  return ERASE_OK;
}

#define HIPCHK(c, call)                                  \
  do {                                                   \
    if (!hip_ok((c), (call), #call)) return ERASE_ERR_HIP; \
  } while (0)

// Algorithmic cost of each launch (see the measurement notes of the design).
struct Cost {
  double flops = 0, bytes = 0;
  int tile_m = 0, tile_n = 0, split = 0, grid = 0;
};

Cost gemm_cost(const GemmDesc& g) {
  Cost c;
  c.tile_m = g.bm;
  c.tile_n = g.bn;
  c.split = g.split;
  c.grid = (int)(cdiv(g.M, g.bm) * cdiv(g.N, g.bn) * g.split);
  return c;
}

class Enqueuer {
 public:
  Enqueuer(Ctx* c, bool timed) : c_(c), timed_(timed) {}

  template <class F>
  erase_status run(int kind, int blk, int layer, int stream_id, hipStream_t s, Cost cost, F&& fn) {
    TimedLaunch tl{};
    LaunchEv lev;
    if (timed_) {
      if (ev_ + 2 > c_->tev.size()) {
        c_->err = "timing event pool exhausted";
        return ERASE_ERR_STATE;
      }
      tl.e0 = c_->tev[ev_++];
      tl.e1 = c_->tev[ev_++];
      lev.e0 = tl.e0;  // stamped at the kernel's own start and end
      lev.e1 = tl.e1;
    }
    (void)s;
    if (!timed_ && end_) {
      lev.e1 = end_;  // recorded at this kernel's end (the last such launch wins)
      end_used_ = true;
    }
    hipError_t e = fn(lev);
    if (!hip_ok(c_, e, "kernel launch")) return ERASE_ERR_HIP;
    if (timed_) {
      tl.rec.kind = kind;
      tl.rec.block = blk;
      tl.rec.layer = layer;
      tl.rec.stream = stream_id;
      tl.rec.flops = cost.flops;
      tl.rec.bytes = cost.bytes;
      tl.rec.tile_m = cost.tile_m;
      tl.rec.tile_n = cost.tile_n;
      tl.rec.split = cost.split;
      tl.rec.grid = cost.grid;
      out_.push_back(tl);
    }
    return ERASE_OK;
  }
  std::vector<TimedLaunch>& launches() { return out_; }
  // Stream-ordering event to be recorded by the launches that follow, at
  // each kernel's end (in place of a record after them, which costs a packet
  // of its own on the stream); none while timing (the launches carry their
  // timing events) or under graph capture.  end_recorded() tells whether a
  // launch took it since set_end.
  void set_end(hipEvent_t e) {
    end_ = ends_ok_ ? e : nullptr;
    end_used_ = false;
  }
  bool end_recorded() const { return end_used_; }
  void no_end_events() { ends_ok_ = false; }

 private:
  Ctx* c_;
  bool timed_;
  bool ends_ok_ = true, end_used_ = false;
  hipEvent_t end_ = nullptr;
  size_t ev_ = 0;
  std::vector<TimedLaunch> out_;
};

#define RUN(...)                                   \
  do {                                             \
    erase_status st_ = q.run(__VA_ARGS__);         \
    if (st_ != ERASE_OK) return st_;               \
  } while (0)

// Input of layer l of block b (row-major).
void layer_input(const Ctx* c, int b, int l, const void* x, int par, const void** mn, int64_t* ldmn) {
  const Plan& P = c->P;
  const BlockRT& B = P.blk[b];
  if (l > 0) {
    *mn = B.layer[l - 1].y;
    *ldmn = B.layer[l - 1].ldy;
  } else if (B.input_src == ERASE_IN_X) {
    if (P.x_in_place) {
      *mn = x;
      *ldmn = c->cfg.x_ld;
    } else {
      *mn = P.xp[par];
      *ldmn = P.ldxp;
    }
  } else {
    const BlockRT& A = P.blk[b - 1];
    const LayerRT& R = A.layer[A.L - 1];
    *mn = R.y;
    *ldmn = R.ldy;
  }
}

erase_status enqueue_head(Ctx* c, Enqueuer& q, int b, const float* labels, hipStream_t s, int sid);

// Block b's forward GEMMs and, unless it is fused into the last GEMM or
// `with_head` is false, its local head and loss.
erase_status enqueue_forward(Ctx* c, Enqueuer& q, int b, const void* x, const float* labels, hipStream_t s, int sid,
                             bool with_head = true, int l_begin = 0, int l_end = -1, int par = -1) {
  const Plan& P = c->P;
  const BlockRT& B = P.blk[b];
  const int M = P.M, esz = P.esz;
  // (the worker thread passes the step parity it was given; c->par may
  // already belong to the next step)
  if (par < 0) par = c->par;
  const void* x0;
  int64_t ldx0;
  layer_input(c, b, 0, x, par, &x0, &ldx0);
  if (l_end < 0) l_end = B.L;
  for (int l = l_begin; l < l_end; ++l) {
    const LayerRT& R = B.layer[l];
    const void* a;
    int64_t lda;
    layer_input(c, b, l, x, par, &a, &lda);
    GemmDesc g{};
    g.A = a;
    g.lda = lda;
    g.B = R.wsh;
    g.ldb = R.ldwsh;
    g.M = M;
    g.N = R.N;
    g.K = (int)roundup(R.K, P.bf16 ? 64 : 32);
    g.kps = R.fwd.kps;
    g.split = 1;
    g.bm = R.fwd.bm;
    g.bn = R.fwd.bn;
    g.group = R.fwd.group;
    g.kgroups = R.fwd.kgroups;
    EpiParams e{};
    e.bias = B.buf.param + R.offb;
    e.y = R.y;
    e.ldy = R.ldy;
    const bool fused = B.head_fused && l == B.L - 1;
    const int kind = R.kind == ERASE_LAYER_CROSS ? GK_FWD_CROSS : fused ? GK_FWD_HEAD : GK_FWD_RELU;
    if (kind == GK_FWD_CROSS) {
      e.x0 = x0;
      e.ldx0 = ldx0;
      e.xl = a;
      e.ldxl = lda;
    }
    Cost cost = gemm_cost(g);
    cost.flops = 2.0 * M * R.N * R.K;
    cost.bytes = double(esz) * (double(M) * R.K + double(R.N) * R.K + double(M) * R.N) + 4.0 * R.N +
                 (kind == GK_FWD_CROSS ? 2.0 * esz * M * R.N : 0.0);
    if (fused) {
      // z leaves the chip only when the next block reads it
      if (!R.needy) e.y = nullptr;
      e.hw = B.buf.param + B.off_w;
      e.hc = B.buf.param + B.off_c;
      e.labels = labels;
      e.lam = B.lam;
      e.inv_m = 1.0f / float(M);
      e.dmn = R.dmn;
      e.lddmn = R.lddmn;
      e.pdw = B.pdw;
      e.pdc = B.pdc;
      e.ploss = B.ploss;
      cost.flops += 4.0 * M * R.N;
      cost.bytes = double(esz) * (double(M) * R.K + double(R.N) * R.K + double(M) * R.N * ((R.needy ? 1 : 0) + 1)) +
                   4.0 * R.N + 4.0 * M + 4.0 * R.N + 4.0 * B.nhead * (R.N + 2);
    }
    const int bf = P.bf16;
    RUN(fused ? 8 : g.kgroups == 2 ? 9 : 1, b, l, sid, s, cost,
        [&](const LaunchEv& ev) { return launch_gemm(bf, kind, g, e, s, ev); });
  }
  if (B.head_fused || !with_head || l_end < B.L) return ERASE_OK;
  return enqueue_head(c, q, b, labels, s, sid);
}

// Standalone local head, loss and loss gradient of block b (Section 2.1).
erase_status enqueue_head(Ctx* c, Enqueuer& q, int b, const float* labels, hipStream_t s, int sid) {
  const Plan& P = c->P;
  const BlockRT& B = P.blk[b];
  const int M = P.M, esz = P.esz;
  const LayerRT& Rl = B.layer[B.L - 1];
  HeadArgs h{};
  h.z = Rl.y;
  h.ldz = Rl.ldy;
  h.w = B.buf.param + B.off_w;
  h.c = B.buf.param + B.off_c;
  h.y = labels;
  h.lam = B.lam;
  h.inv_m = 1.0f / float(M);
  h.M = M;
  h.N = Rl.N;
  h.dmn = Rl.dmn;
  h.lddmn = Rl.lddmn;

  h.pdw = B.pdw;
  h.pdc = B.pdc;
  h.ploss = B.ploss;
  Cost cost;
  cost.grid = B.nhead;
  cost.flops = 4.0 * M * Rl.N;
  cost.bytes = double(esz) * M * Rl.N * (1 + 1 + (Rl.dmn ? 1 : 0)) + 4.0 * M + 4.0 * Rl.N + 4.0 * B.nhead * (Rl.N + 2);
  const int bf = P.bf16;
  RUN(2, b, -1, sid, s, cost, [&](const LaunchEv& ev) { return launch_head(bf, h, s, ev); });
  return ERASE_OK;
}

// Backward GEMMs of block b, last layer first.  Per layer l: the weight and
// bias gradient dW = dH^T a_{l-1}, db = row sums of dH^T, and (l > 0) the
// input gradient of the layer below; the block input is detached (Eq. 1), so
// layer 0 has no input gradient.  When both GEMMs of a layer share a tile
// they go out as one launch.
// Arguments and cost of block b's Adam launch (the parameters not updated by
// a fused weight-gradient launch).
AdamArgs adam_args(const Ctx* c, int b, float* losses, int par, Cost* cost) {
  const Plan& P = c->P;
  const BlockRT& B = P.blk[b];
  AdamArgs a{};
  a.seg = B.segs_dev;
  a.nseg = (int)B.segs.size();
  for (int i = 0; i < a.nseg; ++i) a.chunk0[i] = B.segs[i].chunk0;
  a.nchunks = B.nchunks;
  a.hyper = reinterpret_cast<const float*>(P.t + 2) + 2 * par;
  a.beta1 = c->cfg.beta1;
  a.beta2 = c->cfg.beta2;
  a.eps = c->cfg.eps;
  a.ploss = B.ploss;
  a.nloss = B.nhead;
  a.inv_m = 1.0f / float(P.M);
  a.loss_out = losses + b;
  a.status = P.status;
  cost->grid = (int)B.nchunks;
  for (const AdamSeg& sg : B.segs) {
    const double n = double(sg.rows) * sg.cols;
    cost->flops += 12.0 * n;
    cost->bytes += n * (4.0 * sg.nsplit + 24.0 + (sg.g ? 4.0 : 0.0) + (sg.sh ? P.esz : 0) + (sg.sht ? P.esz : 0));
  }
  return a;
}

// Block b's backward.  With `losses` set, a block whose first-layer weight
// gradient carries the fused Adam update also runs the Adam update of its
// other parameters in that launch (*adam_done = true); the caller then
// launches no separate Adam for the block.
erase_status enqueue_backward(Ctx* c, Enqueuer& q, int b, const void* x, hipStream_t s, int sid, int par,
                              bool send = false, float* losses = nullptr, bool* adam_done = nullptr) {
  if (adam_done) *adam_done = false;
  const Plan& P = c->P;
  const BlockRT& B = P.blk[b];
  const int M = P.M, esz = P.esz, bf = P.bf16;
  const void* x0;
  int64_t ldx0;
  layer_input(c, b, 0, x, par, &x0, &ldx0);
  for (int l = B.L - 1; l >= 0; --l) {
    const LayerRT& R = B.layer[l];
    const void* inmn;
    int64_t ldinmn;
    layer_input(c, b, l, x, par, &inmn, &ldinmn);
    // dW[n][k] = sum over the batch of dH[m][n] a[m][k]: both row-major
    GemmDesc gw{};
    gw.A = R.dmn;
    gw.lda = R.lddmn;
    gw.B = inmn;
    gw.ldb = ldinmn;
    gw.M = R.N;
    gw.N = R.K;
    gw.K = (int)roundup(M, P.bf16 ? 64 : 32);
    gw.kps = R.wgrad.kps;
    gw.split = R.wgrad.split;
    gw.bm = R.wgrad.bm;
    gw.bn = R.wgrad.bn;
    gw.group = R.wgrad.group;
    EpiParams ew{};
    ew.part = R.part;
    ew.ldp = R.ldp;
    ew.pstride = R.pstride;
    ew.bpart = R.bpart;
    Cost cw = gemm_cost(gw);
    cw.flops = 2.0 * M * R.N * R.K;
    cw.bytes = double(esz) * M * (double(R.N) + R.K) + 4.0 * R.wgrad.split * (double(R.N) * R.K + R.N);
    gw.kgroups = R.wgrad.kgroups;
    if (R.fused_adam) {
      ew.ap = B.buf.param + R.offW;
      ew.am = B.buf.m + R.offW;
      ew.av = B.buf.v + R.offW;
      ew.ag = B.buf.grad ? B.buf.grad + R.offW : nullptr;
      ew.ash = R.wsh;
      ew.ldash = R.ldwsh;
      ew.bp = B.buf.param + R.offb;
      ew.bm = B.buf.m + R.offb;
      ew.bv = B.buf.v + R.offb;
      ew.bg = B.buf.grad ? B.buf.grad + R.offb : nullptr;
      ew.hyper = reinterpret_cast<const float*>(P.t + 2) + 2 * par;
      ew.b1 = c->cfg.beta1;
      ew.b2 = c->cfg.beta2;
      ew.eps = c->cfg.eps;
      // no partial slice is stored; Adam's per-parameter traffic moves here
      const double n = double(R.N) * R.K + R.N;
      cw.flops += 12.0 * n;
      cw.bytes += n * (24.0 + (ew.ag ? 4.0 : 0.0)) + double(R.N) * R.K * esz - 4.0 * n;
    }
    if (l == 0) {
      if (losses && R.fused_adam) {
        Cost ca;
        const AdamArgs aa = adam_args(c, b, losses, par, &ca);
        cw.flops += ca.flops;
        cw.bytes += ca.bytes;
        cw.grid += (ca.grid + 1) / 2;
        RUN(11, b, l, sid, s, cw, [&](const LaunchEv& ev) { return launch_wgrad_adam(bf, gw, ew, aa, s, ev); });
        if (adam_done) *adam_done = true;
      } else {
        RUN(gw.kgroups == 2 ? 10 : 3, b, l, sid, s, cw,
            [&](const LaunchEv& ev) { return launch_gemm(bf, GK_WGRAD, gw, ew, s, ev); });
      }
      if (send && B.send) {
        // undetached: the gradient at the block input, dX = dH_0 W_0, is
        // added to the previous block's output gradient (its head's term,
        // already in place) under that block's ReLU mask
        const LayerRT& Rp = P.blk[b - 1].layer[P.blk[b - 1].L - 1];
        GemmDesc gx{};
        gx.A = R.dmn;
        gx.lda = R.lddmn;
        gx.B = R.wsht;
        gx.ldb = R.ldwsht;
        gx.M = M;
        gx.N = R.K;
        gx.K = (int)roundup(R.N, P.bf16 ? 64 : 32);
        gx.kps = R.dgrad.kps;
        gx.split = 1;
        gx.bm = R.dgrad.bm;
        gx.bn = R.dgrad.bn;
        gx.group = R.dgrad.group;
        EpiParams ex{};
        ex.res = Rp.dmn;
        ex.ldres = Rp.lddmn;
        ex.mask = Rp.y;
        ex.ldmask = Rp.ldy;
        ex.below_cross = 0;
        ex.dmn = Rp.dmn;
        ex.lddmn = Rp.lddmn;
        Cost cx = gemm_cost(gx);
        cx.flops = 2.0 * M * R.N * R.K;
        cx.bytes = double(esz) * (double(M) * R.N + double(R.N) * R.K + 3.0 * double(M) * R.K);
        RUN(4, b, l, sid, s, cx, [&](const LaunchEv& ev) { return launch_gemm(bf, GK_DGRAD, gx, ex, s, ev); });
      }
      break;
    }
    const LayerRT& Rb = B.layer[l - 1];
    GemmDesc gd{};
    gd.A = R.dmn;
    gd.lda = R.lddmn;
    gd.B = R.wsht;
    gd.ldb = R.ldwsht;
    gd.M = M;
    gd.N = R.K;
    gd.K = (int)roundup(R.N, P.bf16 ? 64 : 32);
    gd.kps = R.dgrad.kps;
    gd.split = 1;
    gd.bm = R.dgrad.bm;
    gd.bn = R.dgrad.bn;
    gd.group = R.dgrad.group;
    EpiParams ed{};
    if (R.kind == ERASE_LAYER_CROSS) {
      ed.res = R.g;
      ed.ldres = R.ldg;
    }
    ed.dmn = Rb.dmn;
    ed.lddmn = Rb.lddmn;
    if (Rb.kind == ERASE_LAYER_CROSS) {
      ed.below_cross = 1;
      ed.x0 = x0;
      ed.ldx0 = ldx0;
      ed.gout = Rb.g;
      ed.ldgout = Rb.ldg;
    } else {
      ed.below_cross = 0;
      ed.mask = Rb.y;
      ed.ldmask = Rb.ldy;
    }
    Cost cd = gemm_cost(gd);
    cd.flops = 2.0 * M * R.N * R.K;
    const double outs = 1.0 + (ed.gout ? 1.0 : 0.0);
    cd.bytes = double(esz) * (double(M) * R.N + double(R.N) * R.K + double(M) * R.K * (outs + 1.0) +
                              (ed.res ? double(M) * R.K : 0.0));
    if (R.grouped) {
      Cost cg = cd;
      cg.flops += cw.flops;
      cg.bytes += cw.bytes;
      cg.grid += cw.grid;
      cg.split = cw.split;
      RUN(6, b, l, sid, s, cg, [&](const LaunchEv& ev) { return launch_bwd_gemm(bf, gd, ed, gw, ew, s, ev); });
    } else {
      RUN(3, b, l, sid, s, cw, [&](const LaunchEv& ev) { return launch_gemm(bf, GK_WGRAD, gw, ew, s, ev); });
      RUN(4, b, l, sid, s, cd, [&](const LaunchEv& ev) { return launch_gemm(bf, GK_DGRAD, gd, ed, s, ev); });
    }
  }
  return ERASE_OK;
}

erase_status enqueue_adam(Ctx* c, Enqueuer& q, int b, float* losses, hipStream_t s, int sid, int par) {
  const Plan& P = c->P;
  Cost cost;
  const AdamArgs a = adam_args(c, b, losses, par, &cost);
  const int bf = P.bf16;
  RUN(5, b, -1, sid, s, cost, [&](const LaunchEv& ev) { return launch_adam(bf, a, s, ev); });
  return ERASE_OK;
}

// One step's launches.  `sched` selects serial or overlapped order; graph
// schedules call this under stream capture.  With `threaded` (uncaptured,
// untimed, worker dispatch on) the ERASE schedules hand each block's backward
// and Adam to the worker thread, which enqueues them on the backward stream
// while this thread goes on with the next block's forward.
erase_status enqueue_step(Ctx* c, Enqueuer& q, const void* x, const float* labels, int sched, float* losses,
                          bool threaded = false) {
  const Plan& P = c->P;
  const bool pipeline = sched == ERASE_SCHED_PIPELINE;
  const bool adam_end = sched == ERASE_SCHED_OVERLAP_ADAM_END;
  const bool overlap = sched == ERASE_SCHED_OVERLAP || sched == ERASE_SCHED_OVERLAP_GRAPH || pipeline || adam_end;
  const int nb = (int)P.blk.size();
  const int ns = (int)c->sbs.size();
  const int par = c->par;
  hipStream_t sf = c->sf;
  {
    PrologueArgs pa{};
    pa.t = P.t;
    pa.lr = c->cfg.lr;
    pa.beta1 = c->cfg.beta1;
    pa.beta2 = c->cfg.beta2;
    pa.x = x;
    pa.ldx = c->cfg.x_ld;
    pa.hyper = reinterpret_cast<float*>(P.t + 2) + 2 * par;
    pa.xp = P.xp[par];
    pa.ldxp = P.ldxp;

    pa.M = P.M;
    pa.K = c->cfg.in_dim;
    Cost cost;
    cost.bytes = P.xp[0] ? 2.0 * P.esz * double(P.M) * c->cfg.in_dim : 0.0;
    const int bf = P.bf16;
    RUN(0, -1, -1, 0, sf, cost, [&](const LaunchEv& ev) { return launch_prologue(bf, pa, sf, ev); });
  }
  if (overlap) {
    // ERASE: block b's backward and Adam go to backward stream b % ns as soon
    // as its forward and local loss are enqueued; the step ends with the
    // forward stream joined on every backward stream used.
    threaded = threaded && c->worker != nullptr;
    for (int b = 0; b < nb; ++b) {
      const int k = b % ns;
      hipStream_t sb = c->sbs[k];
      const bool chained_next = b + 1 < nb && P.blk[b + 1].input_src == ERASE_IN_PREV;
      if (pipeline && c->pending) {
        // no end-of-step join: block b's forward waits only for the previous
        // step's backward of block b (its weights, its activation buffers)
        // and, in a chain, of block b+1 (which reads block b's output).  With
        // the worker, those backward launches (and their event records) must
        // have been enqueued before this thread waits on the events.
        if (threaded) {
          erase_status st = wait_job(c, c->job_of[b]);
          if (st == ERASE_OK && chained_next) st = wait_job(c, c->job_of[b + 1]);
          if (st != ERASE_OK) return st;
        }
        HIPCHK(c, hipStreamWaitEvent(sf, c->eb[b], 0));
        if (chained_next) HIPCHK(c, hipStreamWaitEvent(sf, c->eb[b + 1], 0));
      }
      // a standalone head goes to the backward stream, in front of the
      // block's backward: the next block's forward waits only for the body.
      // A head fused into the last layer takes that layer with it when no
      // later block reads the block's output.
      const bool head_b = !P.blk[b].head_fused;
      const int L = P.blk[b].L;
      const bool last_b = !head_b && L >= 2 && !chained_next;
      q.set_end(c->ef[b]);
      erase_status st = enqueue_forward(c, q, b, x, labels, sf, 0, !head_b, 0, last_b ? L - 1 : L);
      if (st != ERASE_OK) return st;
      if (!q.end_recorded()) HIPCHK(c, hipEventRecord(c->ef[b], sf));
      q.set_end(nullptr);
      if (threaded) {
        // ef[b] is recorded again only in a later step, after this job has
        // finished (the waits above, or the join below), so the job's wait
        // always binds to this step's record
        hipEvent_t efb = c->ef[b], ebb = c->eb[b];
        c->job_of[b] = c->worker->push([c, b, x, labels, losses, sb, k, par, adam_end, head_b, last_b, L, efb,
                                        ebb]() -> erase_status {
          HIPCHK(c, hipStreamWaitEvent(sb, efb, 0));
          Enqueuer wq(c, false);
          wq.set_end(ebb);
          erase_status s2 = head_b ? enqueue_head(c, wq, b, labels, sb, 1 + k)
                            : last_b ? enqueue_forward(c, wq, b, x, labels, sb, 1 + k, true, L - 1, L, par)
                                     : ERASE_OK;
          if (s2 != ERASE_OK) return s2;
          bool done = false;
          s2 = enqueue_backward(c, wq, b, x, sb, 1 + k, par, false, adam_end ? nullptr : losses, &done);
          if (s2 != ERASE_OK) return s2;
          if (!adam_end && !done) {
            s2 = enqueue_adam(c, wq, b, losses, sb, 1 + k, par);
            if (s2 != ERASE_OK) return s2;
          }
          if (!wq.end_recorded()) HIPCHK(c, hipEventRecord(ebb, sb));
          return ERASE_OK;
        });
        continue;
      }
      HIPCHK(c, hipStreamWaitEvent(sb, c->ef[b], 0));
      q.set_end(c->eb[b]);
      if (head_b) {
        st = enqueue_head(c, q, b, labels, sb, 1 + k);
        if (st != ERASE_OK) return st;
      } else if (last_b) {
        st = enqueue_forward(c, q, b, x, labels, sb, 1 + k, true, L - 1, L, par);
        if (st != ERASE_OK) return st;
      }
      bool done = false;
      st = enqueue_backward(c, q, b, x, sb, 1 + k, par, false, adam_end ? nullptr : losses, &done);
      if (st != ERASE_OK) return st;
      if (!adam_end && !done) {
        st = enqueue_adam(c, q, b, losses, sb, 1 + k, par);
        if (st != ERASE_OK) return st;
      }
      if (!q.end_recorded()) HIPCHK(c, hipEventRecord(c->eb[b], sb));
      q.set_end(nullptr);
    }
    if (threaded && !pipeline) {
      erase_status st = quiesce(c);
      if (st != ERASE_OK) return st;
    }
    if (!pipeline)
      for (int b = std::max(0, nb - ns); b < nb; ++b) HIPCHK(c, hipStreamWaitEvent(sf, c->eb[b], 0));
    if (adam_end) {
      // the optimizer steps once, after every block's backward
      for (int b = 0; b < nb; ++b) {
        erase_status st = enqueue_adam(c, q, b, losses, sf, 0, par);
        if (st != ERASE_OK) return st;
      }
    }
  } else {
    // SERIAL, and the conventional (undetached) baseline: every forward,
    // then one backward from the last block to the first, then Adam
    const bool send = sched == ERASE_SCHED_UNDETACHED || sched == ERASE_SCHED_UNDETACHED_GRAPH;
    for (int b = 0; b < nb; ++b) {
      erase_status st = enqueue_forward(c, q, b, x, labels, sf, 0);
      if (st != ERASE_OK) return st;
    }
    std::vector<char> done(nb, 0);
    for (int b = nb - 1; b >= 0; --b) {
      bool d = false;
      erase_status st = enqueue_backward(c, q, b, x, sf, 0, par, send, losses, &d);
      if (st != ERASE_OK) return st;
      done[b] = d;
    }
    for (int b = 0; b < nb; ++b) {
      if (done[b]) continue;
      erase_status st = enqueue_adam(c, q, b, losses, sf, 0, par);
      if (st != ERASE_OK) return st;
    }
  }
  return ERASE_OK;
}

int launches_per_step(const Plan& P) {
  int n = 1;  // prologue
  for (const BlockRT& B : P.blk) {
    n += B.L + (B.head_fused ? 0 : 1) + 1 + 1;  // forward GEMMs, head, first layer's weight gradient, Adam
    n += B.send ? 1 : 0;                         // undetached: input gradient sent to the previous block
    for (int l = 1; l < B.L; ++l) n += B.layer[l].grouped ? 1 : 2;
  }
  return n;
}

// Join the backward streams of an unjoined PIPELINE step into the forward
// stream (enqueued, not captured).
erase_status join_pending(Ctx* c) {
  if (!c->pending) return ERASE_OK;
  erase_status st = quiesce(c);
  if (st != ERASE_OK) return st;
  for (size_t b = 0; b < c->eb.size(); ++b) HIPCHK(c, hipStreamWaitEvent(c->sf, c->eb[b], 0));
  c->pending = false;
  return ERASE_OK;
}

erase_status refresh(Ctx* c) {
  for (const BlockRT& B : c->P.blk) {
    AdamArgs a{};
    a.seg = B.rsegs_dev;
    a.nseg = (int)B.rsegs.size();
    for (int i = 0; i < a.nseg; ++i) a.chunk0[i] = B.rsegs[i].chunk0;
    a.nchunks = B.rnchunks;
    HIPCHK(c, launch_refresh(c->P.bf16, a, c->sf));
  }
  return ERASE_OK;
}

void destroy_graphs(Ctx* c) {
  for (GraphEntry& g : c->graphs) {
    if (g.exec) (void)hipGraphExecDestroy(g.exec);
    if (g.graph) (void)hipGraphDestroy(g.graph);
  }
  c->graphs.clear();
}

}  // namespace

// The opaque context handle of the C ABI.
struct erase_ctx {
  Ctx impl;
};

namespace {
Ctx* as_ctx(erase_ctx* p) { return p ? &p->impl : nullptr; }
}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

erase_status erase_param_count(const erase_config* cfg, int32_t block, int64_t* count) {
  if (!count) return ERASE_ERR_INVALID_ARG;
  erase_status st = validate(cfg, nullptr);
  if (st != ERASE_OK) return st;
  if (block < 0 || block >= cfg->n_blocks) return ERASE_ERR_INVALID_ARG;
  const erase_block_spec& B = cfg->blocks[block];
  int64_t n = 0;
  for (int l = 0; l < B.n_layers; ++l) n += int64_t(B.layers[l].in_dim) * B.layers[l].out_dim + B.layers[l].out_dim;
  n += B.layers[B.n_layers - 1].out_dim + 1;
  *count = n;
  return ERASE_OK;
}

erase_status erase_workspace_bytes(const erase_config* cfg, size_t* bytes) {
  if (!bytes) return ERASE_ERR_INVALID_ARG;
  erase_status st = validate(cfg, nullptr);
  if (st != ERASE_OK) return st;
  Plan P;
  *bytes = build_plan(*cfg, 0, &P);
  return ERASE_OK;
}

erase_status erase_init(const erase_config* cfg, const erase_block_buffers* bufs, void* workspace, size_t ws_bytes,
                        void* s_fwd, void* s_bwd, erase_ctx** ctx_out) {
  void* const one[1] = {s_bwd};
  return erase_init_streams(cfg, bufs, workspace, ws_bytes, s_fwd, one, 1, ctx_out);
}

erase_status erase_init_streams(const erase_config* cfg, const erase_block_buffers* bufs, void* workspace,
                                size_t ws_bytes, void* s_fwd, void* const* s_bwd, int32_t n_bwd, erase_ctx** ctx_out) {
  if (!ctx_out) return ERASE_ERR_INVALID_ARG;
  *ctx_out = nullptr;
  std::string err;
  erase_status st = validate(cfg, &err);
  if (st != ERASE_OK) return st;
  if (!bufs) return ERASE_ERR_INVALID_ARG;
  for (int b = 0; b < cfg->n_blocks; ++b) {
    if (!bufs[b].param || !bufs[b].m || !bufs[b].v) return ERASE_ERR_INVALID_ARG;
    const uintptr_t al = reinterpret_cast<uintptr_t>(bufs[b].param) | reinterpret_cast<uintptr_t>(bufs[b].m) |
                         reinterpret_cast<uintptr_t>(bufs[b].v) | reinterpret_cast<uintptr_t>(bufs[b].grad);
    if (al % 4) return ERASE_ERR_INVALID_ARG;
  }
  if (!s_fwd || !s_bwd || n_bwd < 1 || n_bwd > kMaxBwdStreams) return ERASE_ERR_INVALID_ARG;
  for (int i = 0; i < n_bwd; ++i) {
    if (!s_bwd[i] || s_bwd[i] == s_fwd) return ERASE_ERR_INVALID_ARG;
    for (int j = 0; j < i; ++j)
      if (s_bwd[j] == s_bwd[i]) return ERASE_ERR_INVALID_ARG;
  }
  if (!workspace || reinterpret_cast<uintptr_t>(workspace) % kAlign) return ERASE_ERR_WORKSPACE;
  {
    Plan probe;
    if (ws_bytes < build_plan(*cfg, 0, &probe)) return ERASE_ERR_WORKSPACE;
  }

  erase_ctx* h = new erase_ctx();
  Ctx* c = &h->impl;
  c->cfg = *cfg;
  c->blocks.assign(cfg->blocks, cfg->blocks + cfg->n_blocks);
  c->layers.resize(cfg->n_blocks);
  for (int b = 0; b < cfg->n_blocks; ++b) {
    c->layers[b].assign(cfg->blocks[b].layers, cfg->blocks[b].layers + cfg->blocks[b].n_layers);
    c->blocks[b].layers = c->layers[b].data();
  }
  c->cfg.blocks = c->blocks.data();
  c->ws = static_cast<char*>(workspace);
  c->ws_bytes = ws_bytes;
  c->sf = static_cast<hipStream_t>(s_fwd);
  for (int i = 0; i < n_bwd; ++i) c->sbs.push_back(static_cast<hipStream_t>(s_bwd[i]));
  build_plan(c->cfg, reinterpret_cast<uintptr_t>(workspace), &c->P);
  build_segments(&c->P, bufs);

  auto bail = [&](erase_status s) {
    for (hipEvent_t e : c->ef) (void)hipEventDestroy(e);
    for (hipEvent_t e : c->eb) (void)hipEventDestroy(e);
    delete h;
    return s;
  };
  if (hipGetDevice(&c->device) != hipSuccess) return bail(ERASE_ERR_HIP);
  // The ordering events only order streams of this device (no host waits on
  // them): recorded without the system-scope fence, which writes back and
  // invalidates the caches at every record
  const unsigned evflags = hipEventDisableTiming | hipEventDisableSystemFence;
  for (int b = 0; b < cfg->n_blocks; ++b) {
    hipEvent_t e1, e2;
    if (hipEventCreateWithFlags(&e1, evflags) != hipSuccess) return bail(ERASE_ERR_HIP);
    c->ef.push_back(e1);
    if (hipEventCreateWithFlags(&e2, evflags) != hipSuccess) return bail(ERASE_ERR_HIP);
    c->eb.push_back(e2);
  }
  // zero the workspace once (counters, and the padding every GEMM operand
  // relies on: nothing writes outside the logical extents afterwards), then
  // the segment tables and the GEMM copies of the weights
  if (hipMemsetAsync(c->ws, 0, c->P.bytes, c->sf) != hipSuccess) return bail(ERASE_ERR_HIP);
  for (BlockRT& B : c->P.blk) {
    if (hipMemcpyAsync(B.segs_dev, B.segs.data(), sizeof(AdamSeg) * B.segs.size(), hipMemcpyHostToDevice, c->sf) !=
            hipSuccess ||
        hipMemcpyAsync(B.rsegs_dev, B.rsegs.data(), sizeof(AdamSeg) * B.rsegs.size(), hipMemcpyHostToDevice,
                       c->sf) != hipSuccess)
      return bail(ERASE_ERR_HIP);
  }
  if (refresh(c) != ERASE_OK) return bail(ERASE_ERR_HIP);
  // the host copies of the segment tables must outlive the async copies:
  // they live in the context, which outlives the stream work it enqueued
  *ctx_out = h;
  return ERASE_OK;
}

erase_status erase_step(erase_ctx* ctx, const void* x, const float* labels, int32_t schedule, float* losses) {
  Ctx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (!x || !labels || !losses) return ERASE_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(x) % 16 || reinterpret_cast<uintptr_t>(labels) % 4 ||
      reinterpret_cast<uintptr_t>(losses) % 4)
    return ERASE_ERR_INVALID_ARG;
  if (schedule < ERASE_SCHED_SERIAL || schedule > ERASE_SCHED_UNDETACHED_GRAPH) return ERASE_ERR_INVALID_ARG;
  if ((schedule == ERASE_SCHED_UNDETACHED || schedule == ERASE_SCHED_UNDETACHED_GRAPH) && !c->P.undet_ok) {
    c->err = "undetached schedule: a chained block must start, and the block it reads must end, with linear+ReLU";
    return ERASE_ERR_UNSUPPORTED;
  }
  const bool graph = schedule == ERASE_SCHED_SERIAL_GRAPH || schedule == ERASE_SCHED_OVERLAP_GRAPH ||
                     schedule == ERASE_SCHED_UNDETACHED_GRAPH;
  if (graph && c->timing) return ERASE_ERR_UNSUPPORTED;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != c->device) {
    c->err = "erase_step called with a different current device than erase_init";
    return ERASE_ERR_STATE;
  }
  const bool erase_order = schedule == ERASE_SCHED_OVERLAP || schedule == ERASE_SCHED_PIPELINE ||
                           schedule == ERASE_SCHED_OVERLAP_ADAM_END;
  const bool threaded = c->use_worker && erase_order && !c->timing;
  // a worker-dispatched PIPELINE step orders itself against the previous
  // step's jobs block by block; everything else starts with the worker idle
  if (!(threaded && schedule == ERASE_SCHED_PIPELINE)) {
    erase_status st = quiesce(c);
    if (st != ERASE_OK) return st;
  }
  c->par = (int)((c->hstep + 1) & 1);
  if (schedule != ERASE_SCHED_PIPELINE) {
    erase_status st = join_pending(c);
    if (st != ERASE_OK) return st;
  }
  if (!graph) {
    Enqueuer q(c, c->timing);
    if (c->timing) {
      HIPCHK(c, hipEventRecord(c->tstart, c->sf));
      HIPCHK(c, hipEventRecord(c->tnull0, c->sf));
      HIPCHK(c, hipEventRecord(c->tnull1, c->sf));
    }
    erase_status st = enqueue_step(c, q, x, labels, schedule, losses, threaded);
    if (st != ERASE_OK) {
      c->sticky = st == ERASE_ERR_HIP ? st : c->sticky;
      return st;
    }
    if (c->timing) {
      c->last = q.launches();
      c->last_valid = true;
    }
    if (schedule == ERASE_SCHED_PIPELINE) c->pending = true;
    c->hstep += 1;
    return ERASE_OK;
  }
  GraphEntry* ge = nullptr;
  for (GraphEntry& g : c->graphs)
    if (g.x == x && g.y == labels && g.losses == losses && g.sched == schedule && g.par == c->par) ge = &g;
  if (!ge) {
    if ((int)c->graphs.size() >= kMaxGraphs) {
      // evict the oldest entry; its replays are ordered before anything new on sf
      HIPCHK(c, hipStreamSynchronize(c->sf));
      GraphEntry old = c->graphs.front();
      if (old.exec) (void)hipGraphExecDestroy(old.exec);
      if (old.graph) (void)hipGraphDestroy(old.graph);
      c->graphs.erase(c->graphs.begin());
    }
    GraphEntry g{x, labels, losses, schedule, c->par, nullptr, nullptr};
    HIPCHK(c, hipStreamBeginCapture(c->sf, hipStreamCaptureModeThreadLocal));
    Enqueuer q(c, false);
    q.no_end_events();
    erase_status st = enqueue_step(c, q, x, labels, schedule, losses);
    hipGraph_t graph_h = nullptr;
    hipError_t ee = hipStreamEndCapture(c->sf, &graph_h);
    if (st != ERASE_OK) {
      if (graph_h) (void)hipGraphDestroy(graph_h);
      return st;
    }
    HIPCHK(c, ee);
    g.graph = graph_h;
    if (!hip_ok(c, hipGraphInstantiate(&g.exec, g.graph, nullptr, nullptr, 0), "hipGraphInstantiate")) {
      (void)hipGraphDestroy(g.graph);
      return ERASE_ERR_HIP;
    }
    c->graphs.push_back(g);
    ge = &c->graphs.back();
  }
  HIPCHK(c, hipGraphLaunch(ge->exec, c->sf));
  c->hstep += 1;
  return ERASE_OK;
}

erase_status erase_sync(erase_ctx* ctx) {
  Ctx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (erase_status q_ = quiesce(c); q_ != ERASE_OK) return q_;
  HIPCHK(c, hipStreamSynchronize(c->sf));
  for (hipStream_t sb : c->sbs) HIPCHK(c, hipStreamSynchronize(sb));
  c->pending = false;
  int status = 0;
  HIPCHK(c, hipMemcpy(&status, c->P.status, sizeof(int), hipMemcpyDeviceToHost));
  if (status != 0) {
    c->sticky = ERASE_ERR_NONFINITE;
    c->err = "a block loss was not finite";
    return ERASE_ERR_NONFINITE;
  }
  return ERASE_OK;
}

erase_status erase_get_step(erase_ctx* ctx, int64_t* t) {
  Ctx* c = as_ctx(ctx);
  if (!c || !t) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (erase_status q_ = quiesce(c); q_ != ERASE_OK) return q_;
  HIPCHK(c, hipStreamSynchronize(c->sf));
  for (hipStream_t sb : c->sbs) HIPCHK(c, hipStreamSynchronize(sb));
  c->pending = false;
  HIPCHK(c, hipMemcpy(t, c->P.t, sizeof(int64_t), hipMemcpyDeviceToHost));
  return ERASE_OK;
}

erase_status erase_set_step(erase_ctx* ctx, int64_t t) {
  Ctx* c = as_ctx(ctx);
  if (!c || t < 0) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (erase_status q_ = quiesce(c); q_ != ERASE_OK) return q_;
  HIPCHK(c, hipStreamSynchronize(c->sf));
  for (hipStream_t sb : c->sbs) HIPCHK(c, hipStreamSynchronize(sb));
  c->pending = false;
  HIPCHK(c, hipMemcpy(c->P.t, &t, sizeof(int64_t), hipMemcpyHostToDevice));
  c->hstep = t;
  return ERASE_OK;
}

erase_status erase_refresh_weights(erase_ctx* ctx) {
  Ctx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (erase_status q_ = quiesce(c); q_ != ERASE_OK) return q_;
  erase_status st = join_pending(c);
  if (st != ERASE_OK) return st;
  return refresh(c);
}

erase_status erase_set_timing(erase_ctx* ctx, int32_t enable) {
  Ctx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (erase_status q_ = quiesce(c); q_ != ERASE_OK) return q_;
  if (enable && c->tev.empty()) {
    const int n = 2 * launches_per_step(c->P);
    for (int i = 0; i < n; ++i) {
      hipEvent_t e;
      HIPCHK(c, hipEventCreate(&e));
      c->tev.push_back(e);
    }
    HIPCHK(c, hipEventCreate(&c->tstart));
    HIPCHK(c, hipEventCreate(&c->tnull0));
    HIPCHK(c, hipEventCreate(&c->tnull1));
  }
  c->timing = enable != 0;
  c->last_valid = false;
  return ERASE_OK;
}

erase_status erase_read_timing(erase_ctx* ctx, erase_kernel_time* out, int32_t cap, int32_t* n) {
  Ctx* c = as_ctx(ctx);
  if (!c || !n || (cap > 0 && !out)) return ERASE_ERR_INVALID_ARG;
  if (!c->last_valid) return ERASE_ERR_STATE;
  *n = (int32_t)c->last.size() + 1;
  if (cap > 0) {  // record 0: the empty interval (kind 7), i.e. the cost of an event pair
    float a = 0.f, b = 0.f;
    HIPCHK(c, hipEventElapsedTime(&a, c->tstart, c->tnull0));
    HIPCHK(c, hipEventElapsedTime(&b, c->tstart, c->tnull1));
    erase_kernel_time r{};
    r.kind = 7;
    r.block = -1;
    r.layer = -1;
    r.start_ms = a;
    r.end_ms = b;
    out[0] = r;
  }
  for (int i = 0; i < (int)c->last.size() && i + 1 < cap; ++i) {
    TimedLaunch& t = c->last[i];
    float a = 0.f, b = 0.f;
    HIPCHK(c, hipEventElapsedTime(&a, c->tstart, t.e0));
    HIPCHK(c, hipEventElapsedTime(&b, c->tstart, t.e1));
    out[i + 1] = t.rec;
    out[i + 1].start_ms = a;
    out[i + 1].end_ms = b;
  }
  return ERASE_OK;
}

erase_status erase_set_dispatch(erase_ctx* ctx, int32_t mode) {
  Ctx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (mode != ERASE_DISPATCH_CALLER && mode != ERASE_DISPATCH_WORKER) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (erase_status q_ = quiesce(c); q_ != ERASE_OK) return q_;
  if (mode == ERASE_DISPATCH_WORKER && !c->worker) {
    try {
      c->worker.reset(new Worker(c->device));
    } catch (...) {
      c->err = "could not start the dispatch thread";
      return ERASE_ERR_STATE;
    }
    c->job_of.assign(c->P.blk.size(), 0);
  }
  c->use_worker = mode == ERASE_DISPATCH_WORKER;
  return ERASE_OK;
}

erase_status erase_embed_bags(const erase_bag_config* cfg, const float* dense, const int64_t* offsets,
                              const int32_t* indices, const float* tables, void* x, int32_t* status,
                              void* stream) {
  if (!cfg) return ERASE_ERR_INVALID_ARG;
  const erase_bag_config& b = *cfg;
  if (b.dtype != ERASE_F32 && b.dtype != ERASE_BF16) return ERASE_ERR_INVALID_ARG;
  const int esz = b.dtype == ERASE_BF16 ? 2 : 4;
  if (b.batch < 1 || b.batch > kMaxBatch || b.n_dense < 0 || b.n_dense > 4096 || b.n_tables < 1 ||
      b.n_tables > 4096 || int64_t(b.n_tables) * b.batch >= (int64_t(1) << 31) || b.dim < 4 || b.dim > 256 ||
      b.dim % 4 || b.rows < 1 || b.rows >= (int64_t(1) << 31) || b.nnz < 0 || b.nnz >= (int64_t(1) << 31) ||
      b.x_ld < int64_t(b.n_dense) + int64_t(b.n_tables) * b.dim || (b.x_ld * esz) % 16)
    return ERASE_ERR_SHAPE;
  auto mis = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a != 0; };
  if ((b.n_dense > 0 && (!dense || mis(dense, 4))) || !offsets || mis(offsets, 8) ||
      (b.nnz > 0 && (!indices || mis(indices, 4))) || !tables || mis(tables, 16) || !x || mis(x, 16) ||
      (status && mis(status, 4)))
    return ERASE_ERR_INVALID_ARG;
  EmbedArgs a{};
  a.dense = dense;
  a.offsets = offsets;
  a.indices = indices;
  a.tables = tables;
  a.x = x;
  a.ldx = b.x_ld;
  a.status = status;
  a.nnz = b.nnz;
  a.rows = b.rows;
  a.M = b.batch;
  a.n_dense = b.n_dense;
  a.T = b.n_tables;
  a.dim = b.dim;
  if (launch_embed_bags(b.dtype == ERASE_BF16, a, static_cast<hipStream_t>(stream)) != hipSuccess)
    return ERASE_ERR_HIP;
  return ERASE_OK;
}

erase_status erase_embed_bags_backward_scratch_bytes(const erase_bag_config* cfg, size_t* bytes) {
  if (!cfg || !bytes) return ERASE_ERR_INVALID_ARG;
  const erase_bag_config& b = *cfg;
  if (b.n_tables < 1 || b.rows < 1 || b.nnz < 0 || int64_t(b.n_tables) * b.rows >= (int64_t(1) << 31) ||
      b.nnz >= (int64_t(1) << 31))
    return ERASE_ERR_SHAPE;
  const int64_t tr = int64_t(b.n_tables) * b.rows;
  const int64_t nr = roundup(std::max<int64_t>(b.nnz, 1), 64);
  *bytes = size_t(4) * size_t(2 * roundup(tr, 64) + 6 * nr + 64 + 2 * roundup(tr / 4096 + 1, 64));
  return ERASE_OK;
}

}  // extern "C"

namespace {

// Shapes and pointers of the embedding-bag backward; *need = its scratch bytes.
erase_status check_bags_backward(const erase_bag_config* cfg, const int64_t* offsets, const int32_t* indices,
                                 const void* dx, const float* table_grad, const int32_t* status, size_t* need) {
  if (!cfg) return ERASE_ERR_INVALID_ARG;
  const erase_bag_config& b = *cfg;
  if (b.dtype != ERASE_F32 && b.dtype != ERASE_BF16) return ERASE_ERR_INVALID_ARG;
  const int esz = b.dtype == ERASE_BF16 ? 2 : 4;
  if (b.batch < 1 || b.batch > kMaxBatch || b.n_dense < 0 || b.n_dense > 4096 || b.n_tables < 1 ||
      b.n_tables > 4096 || int64_t(b.n_tables) * b.batch >= (int64_t(1) << 31) || b.dim < 4 || b.dim > 256 ||
      b.dim % 4 || b.rows < 1 || int64_t(b.n_tables) * b.rows >= (int64_t(1) << 31) || b.nnz < 0 ||
      b.nnz >= (int64_t(1) << 31) || b.x_ld < int64_t(b.n_dense) + int64_t(b.n_tables) * b.dim ||
      (b.x_ld * esz) % 16)
    return ERASE_ERR_SHAPE;
  (void)erase_embed_bags_backward_scratch_bytes(cfg, need);
  auto mis = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a != 0; };
  if (!offsets || mis(offsets, 8) || (b.nnz > 0 && (!indices || mis(indices, 4))) || !dx || mis(dx, 16) ||
      !table_grad || mis(table_grad, 16) || (status && mis(status, 4)))
    return ERASE_ERR_INVALID_ARG;
  return ERASE_OK;
}

// Carve `scratch` (checked) and enqueue the backward's launches.
erase_status run_bags_backward(const erase_bag_config& b, const int64_t* offsets, const int32_t* indices,
                               const void* dx, float* table_grad, void* scratch, int32_t* status, void* stream) {
  const int64_t tr = int64_t(b.n_tables) * b.rows, trr = roundup(tr, 64), nr = roundup(std::max<int64_t>(b.nnz, 1), 64);
  int32_t* w = static_cast<int32_t*>(scratch);
  EmbedBwdArgs a{};
  a.offsets = offsets;
  a.indices = indices;
  a.dx = dx;
  a.lddx = b.x_ld;
  a.grad = table_grad;
  // count and start per table row; bucket, row, owner, slot, and the lists
  // of large and of small rows per entry; the lists' counters; two scan
  // totals per 4096 rows
  a.count = w;
  a.start = w + trr;
  a.bucket = w + 2 * trr;
  a.gid = w + 2 * trr + nr;
  a.owner = w + 2 * trr + 2 * nr;
  a.large = w + 2 * trr + 3 * nr;
  a.slot = w + 2 * trr + 4 * nr;
  a.small = w + 2 * trr + 5 * nr;
  a.nlarge = w + 2 * trr + 6 * nr;
  a.bsum = a.nlarge + 64;
  a.bsum2 = a.bsum + roundup(tr / 4096 + 1, 64);
  a.status = status;
  a.nnz = b.nnz;
  a.trows = tr;
  a.rows = (int)b.rows;
  a.M = b.batch;
  a.n_dense = b.n_dense;
  a.T = b.n_tables;
  a.dim = b.dim;
  if (launch_embed_bags_backward(b.dtype == ERASE_BF16, a, static_cast<hipStream_t>(stream)) != hipSuccess)
    return ERASE_ERR_HIP;
  return ERASE_OK;
}

}  // namespace

extern "C" {

erase_status erase_embed_bags_backward(const erase_bag_config* cfg, const int64_t* offsets, const int32_t* indices,
                                       const void* dx, float* table_grad, void* scratch, size_t scratch_bytes,
                                       int32_t* status, void* stream) {
  size_t need = 0;
  if (erase_status st = check_bags_backward(cfg, offsets, indices, dx, table_grad, status, &need); st != ERASE_OK)
    return st;
  if (!scratch || reinterpret_cast<uintptr_t>(scratch) % 16 || scratch_bytes < need) return ERASE_ERR_WORKSPACE;
  return run_bags_backward(*cfg, offsets, indices, dx, table_grad, scratch, status, stream);
}

erase_status erase_embed_bags_backward_noalloc(const erase_bag_config* cfg, const int64_t* offsets,
                                               const int32_t* indices, const void* dx, float* table_grad,
                                               int32_t* status, void* stream) {
  size_t need = 0;
  if (erase_status st = check_bags_backward(cfg, offsets, indices, dx, table_grad, status, &need); st != ERASE_OK)
    return st;
  if (need > ERASE_BAG_SCRATCH_MAX) return ERASE_ERR_WORKSPACE;
  void* scratch = nullptr;
  size_t bytes = 0;
  if (bag_scratch_device_ptr(&scratch, &bytes) != hipSuccess || bytes < need) return ERASE_ERR_HIP;
  return run_bags_backward(*cfg, offsets, indices, dx, table_grad, scratch, status, stream);
}

erase_status erase_destroy(erase_ctx* ctx) {
  Ctx* c = as_ctx(ctx);
  if (!c) return ERASE_OK;
  if (c->worker) {
    c->worker->drain();
    c->worker.reset();
  }
  (void)hipStreamSynchronize(c->sf);
  for (hipStream_t sb : c->sbs) (void)hipStreamSynchronize(sb);
  destroy_graphs(c);
  for (hipEvent_t e : c->ef) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->eb) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->tev) (void)hipEventDestroy(e);
  if (c->tstart) (void)hipEventDestroy(c->tstart);
  if (c->tnull0) (void)hipEventDestroy(c->tnull0);
  if (c->tnull1) (void)hipEventDestroy(c->tnull1);
  delete ctx;
  return ERASE_OK;
}

const char* erase_status_str(int32_t s) {
  switch (s) {
    case ERASE_OK: return "ok";
    case ERASE_ERR_INVALID_ARG: return "invalid argument";
    case ERASE_ERR_SHAPE: return "invalid shape";
    case ERASE_ERR_UNSUPPORTED: return "unsupported";
    case ERASE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case ERASE_ERR_HIP: return "HIP runtime error";
    case ERASE_ERR_STATE: return "context in a failed state or call out of order";
    case ERASE_ERR_NONFINITE: return "non-finite loss";
    default: return "unknown status";
  }
}

const char* erase_last_error(erase_ctx* ctx) {
  Ctx* c = as_ctx(ctx);
  return c ? c->err.c_str() : "";
}

}  // extern "C"
