// C-ABI entry points of the detached small-transformer step: host
// validation, workspace layout, GEMM plans and the two-stream schedule.
//
// Every layer is a detached block (Eq. 1) with its own next-token head and
// loss (Eq. 2).  ERASE (Section 2.2): block b's backward and update depend
// only on its forward and local loss, so they are launched on a second
// stream as soon as the block's body has run on the forward stream; the head
// (the vocabulary GEMM, the largest launch of a block) goes with them, so
// the forward stream holds only the block bodies that the next block waits
// for.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "erase_tf.h"
#include "internal.h"

namespace {

using namespace erase;

constexpr size_t kAlign = 256;
constexpr int kMaxLayers = 64;
constexpr int64_t kMaxTokens = int64_t(1) << 24;

int64_t rup(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
int64_t cdv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// weights of a block in flat order after the embedding
enum { WQKV = 0, WO = 1, W1 = 2, W2 = 3, WH = 4, NW = 5 };

struct Dims {
  int V = 0, d = 0, H = 0, L = 0, T = 0, B = 0;
  int64_t N = 0, Np = 0;  // positions, rows of every activation buffer
  int64_t rows[NW] = {}, cols[NW] = {};
};

Dims dims_of(const erase_tf_config& c) {
  Dims D;
  D.V = c.vocab;
  D.d = c.d_model;
  D.H = c.n_heads;
  D.L = c.n_layers;
  D.T = c.seq_len;
  D.B = c.batch;
  D.N = int64_t(c.batch) * c.seq_len;
  D.Np = rup(D.N, 128);
  const int64_t d = D.d;
  const int64_t r[NW] = {3 * d, d, 4 * d, d, D.V}, k[NW] = {d, d, d, 4 * d, d};
  for (int i = 0; i < NW; ++i) {
    D.rows[i] = r[i];
    D.cols[i] = k[i];
  }
  return D;
}

erase_status validate(const erase_tf_config* c, std::string* err) {
  if (!c) return ERASE_ERR_INVALID_ARG;
  auto bad = [&](erase_status s, const char* m) {
    if (err) *err = m;
    return s;
  };
  if (c->n_layers < 1 || c->n_layers > kMaxLayers) return bad(ERASE_ERR_SHAPE, "n_layers must be 1..64");
  if (c->n_heads < 1 || c->d_model != 64 * c->n_heads || c->d_model > 4096)
    return bad(ERASE_ERR_SHAPE, "d_model must be 64 * n_heads and at most 4096 (head size 64)");
  if (c->vocab < 64 || c->vocab % 64 || c->vocab > (1 << 20))
    return bad(ERASE_ERR_SHAPE, "vocab must be a multiple of 64 in 64..2^20");
  if (c->seq_len < 1 || c->batch < 1 || int64_t(c->seq_len) * c->batch > kMaxTokens)
    return bad(ERASE_ERR_SHAPE, "batch * seq_len must be 1..2^24");
  if (int64_t(c->seq_len) + 1 > INT32_MAX / std::max(1, c->batch))
    return bad(ERASE_ERR_SHAPE, "batch * (seq_len + 1) exceeds int32");
  const float h[5] = {c->lr, c->beta1, c->beta2, c->eps, c->lambda};
  for (float v : h)
    if (!std::isfinite(v)) return bad(ERASE_ERR_INVALID_ARG, "non-finite hyper-parameter");
  if (c->lr < 0 || c->beta1 < 0 || c->beta1 >= 1 || c->beta2 < 0 || c->beta2 >= 1 || c->eps < 0)
    return bad(ERASE_ERR_INVALID_ARG, "Adam hyper-parameters out of range");
  return ERASE_OK;
}

int64_t param_count(const Dims& D, int b) {
  int64_t n = b == 0 ? int64_t(D.V) * D.d : 0;
  for (int i = 0; i < NW; ++i) n += D.rows[i] * D.cols[i];
  return n;
}

// Workgroup tile and contraction split of one GEMM: the largest tile giving
// at least 384 workgroups (1.5 per CU), else 64x64; weight gradients (fp32
// partial slices reduced by Adam) split the contraction until they reach it.
struct Plan1 {
  int bm = 64, bn = 64, split = 1, kps = 0;
};
Plan1 choose(int64_t M, int64_t N, int64_t K, bool wgrad) {
  Plan1 p;
  const int64_t target = 384;
  auto wgs = [&](int bm, int bn) { return cdv(M, bm) * cdv(N, bn); };
  const int tiles[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
  bool done = false;
  for (auto& t : tiles)
    if (!done && wgs(t[0], t[1]) >= target) {
      p.bm = t[0];
      p.bn = t[1];
      done = true;
    }
  if (!done && wgrad) {
    int s = 1;
    while (s < 16 && wgs(64, 64) * s < target && K / (s * 2) >= 256) s *= 2;
    p.split = s;
  }
  p.kps = (int)rup(cdv(std::max<int64_t>(K, 1), p.split), 64);
  p.split = (int)cdv(std::max<int64_t>(K, 1), p.kps);
  return p;
}

// Forward GEMMs: outputs at least 2048 wide (MLP up-projection, vocabulary
// logits) take 64x128 tiles, three workgroups per CU instead of two 128x128
// (measured on the 16384-row shapes: logits 1.10 vs 1.20 ms, MLP-up 87 vs
// 97 us; the 512-wide outputs are faster with 128x128).
Plan1 choose_fwd(int64_t M, int64_t N, int64_t K) {
  Plan1 p = choose(M, N, K, false);
  if (N >= 2048 && p.bm == 128 && p.bn == 128) p.bm = 64;
  return p;
}

// The vocabulary logits run in 256 x 256 tiles with per-128-column row sums
// when the positions and the vocabulary are multiples of 256 and the width a
// multiple of 64 (the k-step); otherwise in the GEMM core's tiles.
bool logits_wide(const Dims& D) { return D.N % 256 == 0 && D.V % 256 == 0 && D.d % 64 == 0; }

struct Carver {
  uintptr_t base;
  size_t off = kAlign;  // header: step counter, status word, Adam factors
  void* take(size_t n) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    void* p = reinterpret_cast<void*>(base + off);
    off += std::max<size_t>(n, 1);
    return p;
  }
};

struct Lin {
  GemmDesc g{};
  EpiParams e{};
  int kind = 0;
};

struct Block {
  int64_t offw[NW] = {};
  int64_t off_emb = -1;
  uint16_t* sh[NW] = {};   // bf16 copy [rup(rows,128)][cols]
  uint16_t* sht[NW] = {};  // bf16 transposed copy [rup(cols,128)][rows]
  uint16_t* cemb = nullptr;
  float* part[NW] = {};
  Plan1 wp[NW];
  // activations (rows Np, pitch: multiples of 128 elements)
  // logits: the head's exponentials relative to the target logit, then
  // (after tf_head_norm) the head's output gradient up to a row scale
  uint16_t *a0 = nullptr, *n1, *qkv, *o, *a1, *n2, *u, *g, *z, *hn, *logits, *hns;
  uint16_t *dhn, *dz, *du, *dn2, *da1, *dout, *dqkv, *dn1 = nullptr;
  float *r1, *r2, *r3, *lse, *dsum, *lstat, *xref, *rowscale, *rowloss, *ploss, *da0 = nullptr, *gemb = nullptr;
  int32_t* flag = nullptr;
  int ntiles = 0, nloss = 0;
  Lin fwd[NW], dgr[NW], wgr[NW];
  bool grouped[NW] = {};  // input- and weight-gradient GEMMs of the weight in one launch
  std::vector<AdamSeg> segs;
  AdamSeg* segs_dev = nullptr;
  int64_t nchunks = 0;
  erase_block_buffers buf{};
};

struct Layout {
  Dims D;
  int64_t ldd = 0, ld3 = 0, ld4 = 0, ldv = 0;
  int64_t* t = nullptr;
  int* status = nullptr;
  float* hyper = nullptr;
  int32_t *target = nullptr, *input = nullptr, *count = nullptr, *start = nullptr, *fill = nullptr,
          *bucket = nullptr;
  std::vector<Block> blk;
  size_t bytes = 0;
};

size_t build_layout(const erase_tf_config& c, uintptr_t base, Layout* P) {
  Dims D = dims_of(c);
  P->D = D;
  Carver cv{base};
  P->t = reinterpret_cast<int64_t*>(base);
  P->status = reinterpret_cast<int*>(base + 8);
  P->hyper = reinterpret_cast<float*>(base + 16);
  const int64_t Np = D.Np, d = D.d;
  P->ldd = rup(d, 128);
  P->ld3 = rup(3 * d, 128);
  P->ld4 = rup(4 * d, 128);
  P->ldv = rup(D.V, 128);
  auto bf = [&](int64_t rows, int64_t ld) { return static_cast<uint16_t*>(cv.take(size_t(rows * ld) * 2)); };
  auto f32 = [&](int64_t n) { return static_cast<float*>(cv.take(size_t(n) * 4)); };
  auto i32 = [&](int64_t n) { return static_cast<int32_t*>(cv.take(size_t(n) * 4)); };
  P->target = i32(Np);
  P->input = i32(Np);
  P->count = i32(D.V);
  P->start = i32(D.V);
  P->fill = i32(D.V);
  P->bucket = i32(Np);
  P->blk.assign(D.L, Block{});
  const int64_t BHT = int64_t(D.B) * D.H * D.T;
  for (int b = 0; b < D.L; ++b) {
    Block& B = P->blk[b];
    int64_t off = 0;
    if (b == 0) {
      B.off_emb = 0;
      off = int64_t(D.V) * d;
      B.cemb = bf(D.V, d);
      B.a0 = bf(Np, P->ldd);
      B.dn1 = bf(Np, P->ldd);
      B.da0 = f32(Np * P->ldd);
      B.gemb = f32(int64_t(D.V) * d);
    } else {
      B.a0 = P->blk[b - 1].z;
    }
    for (int i = 0; i < NW; ++i) {
      B.offw[i] = off;
      off += D.rows[i] * D.cols[i];
      B.sh[i] = bf(rup(D.rows[i], 128), D.cols[i]);
      B.sht[i] = bf(rup(D.cols[i], 128), D.rows[i]);
    }
    B.n1 = bf(Np, P->ldd);
    B.qkv = bf(Np, P->ld3);
    B.o = bf(Np, P->ldd);
    B.a1 = bf(Np, P->ldd);
    B.n2 = bf(Np, P->ldd);
    B.u = bf(Np, P->ld4);
    B.g = bf(Np, P->ld4);
    B.z = bf(Np, P->ldd);
    B.hn = bf(Np, P->ldd);
    B.logits = bf(Np, P->ldv);
    B.hns = bf(Np, P->ldd);
    B.dhn = bf(Np, P->ldd);
    B.dz = bf(Np, P->ldd);
    B.du = bf(Np, P->ld4);
    B.dn2 = bf(Np, P->ldd);
    B.da1 = bf(Np, P->ldd);
    B.dout = bf(Np, P->ldd);
    B.dqkv = bf(Np, P->ld3);
    B.r1 = f32(Np);
    B.r2 = f32(Np);
    B.r3 = f32(Np);
    B.lse = f32(BHT);
    B.dsum = f32(BHT);
    const Plan1 ph = choose_fwd(D.N, D.V, d);
    B.ntiles = (int)cdv(D.V, logits_wide(D) ? 128 : ph.bn);
    B.lstat = f32(Np * B.ntiles);
    B.xref = f32(Np);
    B.rowscale = f32(Np);
    B.rowloss = f32(Np);
    B.flag = i32(Np);  // zero from init; tf_head_fix clears what it sets
    B.nloss = (int)cdv(D.N, 4);
    B.ploss = f32(B.nloss);
    for (int i = 0; i < NW; ++i) {
      B.wp[i] = choose(D.rows[i], D.cols[i], rup(D.N, 64), true);
      B.part[i] = f32(int64_t(B.wp[i].split) * D.rows[i] * D.cols[i]);
    }
    B.segs_dev = static_cast<AdamSeg*>(cv.take(sizeof(AdamSeg) * (NW + 1)));
  }
  P->bytes = cv.off;
  return cv.off;
}

GemmDesc gdesc(const void* A, int64_t lda, const void* Bm, int64_t ldb, int64_t M, int64_t N, int64_t K,
               const Plan1& p) {
  GemmDesc g{};
  g.A = A;
  g.lda = lda;
  g.B = Bm;
  g.ldb = ldb;
  g.M = (int)M;
  g.N = (int)N;
  g.K = (int)rup(K, 64);
  g.kps = p.kps ? p.kps : g.K;
  g.split = p.split;
  g.bm = p.bm;
  g.bn = p.bn;
  g.group = 0;
  g.kgroups = 1;
  return g;
}

// GEMM launches of every block, fixed at init
bool kg2_pair(int w) { return w == WH; }

void build_gemms(const erase_tf_config& c, Layout* P) {
  const Dims& D = P->D;
  const int64_t N = D.N, d = D.d, V = D.V;
  for (int b = 0; b < D.L; ++b) {
    Block& B = P->blk[b];
    auto fwd = [&](int w, const void* A, int64_t lda, int kind, void* y, int64_t ldy) {
      Lin& L = B.fwd[w];
      L.kind = kind;
      L.g = gdesc(A, lda, B.sh[w], D.cols[w], N, D.rows[w], D.cols[w], choose_fwd(N, D.rows[w], D.cols[w]));
      L.e = EpiParams{};
      L.e.y = y;
      L.e.ldy = ldy;
    };
    fwd(WQKV, B.n1, P->ldd, GK_FWD_LIN, B.qkv, P->ld3);
    fwd(WO, B.o, P->ldd, GK_FWD_LIN, B.a1, P->ldd);
    B.fwd[WO].e.res = B.a0;
    B.fwd[WO].e.ldres = P->ldd;
    fwd(W1, B.n2, P->ldd, GK_FWD_GELU, B.g, P->ld4);
    B.fwd[W1].e.gout = B.u;
    B.fwd[W1].e.ldgout = P->ld4;
    fwd(W2, B.g, P->ld4, GK_FWD_LIN, B.z, P->ldd);
    B.fwd[W2].e.res = B.a1;
    B.fwd[W2].e.ldres = P->ldd;
    fwd(WH, B.hn, P->ldd, GK_FWD_LOGITS, B.logits, P->ldv);
    // GEMM-core tiles (64 x 128): groups of 8 M-tiles (512 positions), each
    // walking every vocabulary tile, keep the tiles an XCD runs at once on
    // about 2 MB of operands (its L2 holds 4 MB).  Measured at 16384 x 32768
    // x 512: 0.89 ms, against 0.99 ms for the generic choice (groups of 128
    // M-tiles, 6 MB of head input in flight per XCD), 0.91 for 16, 0.93 for
    // 2, 1.20 for 1.
    B.fwd[WH].g.group = 8;
    if (logits_wide(D)) {
      B.fwd[WH].g.bm = 256;
      B.fwd[WH].g.bn = 256;
    }
    B.fwd[WH].e.lstat = B.lstat;
    B.fwd[WH].e.ldlstat = B.ntiles;
    B.fwd[WH].e.xref = B.xref;

    // input gradients: A = the output gradient [N][rows], B = transposed copy [cols][rows]
    auto dgr = [&](int w, const void* A, int64_t lda, int kind, void* out, int64_t ldo) {
      Lin& L = B.dgr[w];
      L.kind = kind;
      L.g = gdesc(A, lda, B.sht[w], D.rows[w], N, D.cols[w], D.rows[w], choose_fwd(N, D.cols[w], D.rows[w]));
      L.e = EpiParams{};
      L.e.dmn = out;
      L.e.lddmn = ldo;
    };
    dgr(WH, B.logits, P->ldv, GK_DGRAD, B.dhn, P->ldd);
    dgr(W2, B.dz, P->ldd, GK_DGRAD_GELU, B.du, P->ld4);
    B.dgr[W2].e.mask = B.u;
    B.dgr[W2].e.ldmask = P->ld4;
    dgr(W1, B.du, P->ld4, GK_DGRAD, B.dn2, P->ldd);
    dgr(WO, B.da1, P->ldd, GK_DGRAD, B.dout, P->ldd);
    if (b == 0) dgr(WQKV, B.dqkv, P->ld3, GK_DGRAD, B.dn1, P->ldd);

    // weight gradients: k-major A = output gradient [N][rows], B = layer input [N][cols]
    auto wgr = [&](int w, const void* A, int64_t lda, const void* X, int64_t ldx) {
      Lin& L = B.wgr[w];
      L.kind = GK_WGRAD;
      L.g = gdesc(A, lda, X, ldx, D.rows[w], D.cols[w], N, B.wp[w]);
      L.e = EpiParams{};
      L.e.part = B.part[w];
      L.e.ldp = D.cols[w];
      L.e.pstride = D.rows[w] * D.cols[w];
    };
    wgr(WH, B.logits, P->ldv, B.hns, P->ldd);  // hns: the row-scaled head input
    wgr(W2, B.dz, P->ldd, B.g, P->ld4);
    wgr(W1, B.du, P->ld4, B.n2, P->ldd);
    wgr(WO, B.da1, P->ldd, B.o, P->ldd);
    wgr(WQKV, B.dqkv, P->ld3, B.n1, P->ldd);
    // both gradient GEMMs of a weight read the same output gradient: one
    // launch when they can share a tile (the grouped kernel takes the plain
    // input-gradient epilogue only; a 64x64 weight gradient pulls its
    // input-gradient GEMM down to 64x64)
    for (int w = 0; w < NW; ++w) {
      if (B.dgr[w].g.M == 0 || B.dgr[w].kind != GK_DGRAD) continue;
      GemmDesc& gd = B.dgr[w].g;
      GemmDesc& gw = B.wgr[w].g;
      if (gd.bm == gw.bm && gd.bn == gw.bn && (gd.bm == 128 || gd.bm == 64) && gd.bm == gd.bn) {
        B.grouped[w] = true;
      } else if (gw.bm == 64 && gw.bn == 64) {
        gd.bm = gd.bn = 64;
        B.grouped[w] = true;
      }
      // 128x128 pairs: 512-thread workgroups, two k-groups of four waves
      if (B.grouped[w] && gd.bm == 128 && kg2_pair(w)) gd.kgroups = gw.kgroups = 2;
    }
    (void)V;
    (void)c;
  }
}

void build_segments(Layout* P, const erase_block_buffers* bufs) {
  const Dims& D = P->D;
  for (int b = 0; b < D.L; ++b) {
    Block& B = P->blk[b];
    B.buf = bufs[b];
    B.segs.clear();
    int64_t chunk = 0;
    auto add = [&](int64_t off, int64_t rows, int64_t cols, const float* part, int nsplit, void* sh, void* sht) {
      AdamSeg s{};
      s.p = B.buf.param + off;
      s.m = B.buf.m + off;
      s.v = B.buf.v + off;
      s.g = B.buf.grad ? B.buf.grad + off : nullptr;
      s.part = part;
      s.pstride = rows * cols;
      s.rows = (int)rows;
      s.cols = (int)cols;
      s.ldpart = (int)cols;
      s.nsplit = nsplit;
      s.sh = sh;
      s.ldsh = cols;
      s.sht = sht;
      s.ldsht = rows;
      s.tcols = (int)cdv(cols, ADAM_TC);
      s.chunk0 = chunk;
      chunk += cdv(rows, ADAM_TR) * s.tcols;
      B.segs.push_back(s);
    };
    if (b == 0) add(0, D.V, D.d, B.gemb, 1, B.cemb, nullptr);
    for (int i = 0; i < NW; ++i) add(B.offw[i], D.rows[i], D.cols[i], B.part[i], B.wp[i].split, B.sh[i], B.sht[i]);
    B.nchunks = chunk;
  }
}

struct Rec {
  erase_kernel_time r;
  hipEvent_t e0, e1;
};

struct TfCtx {
  erase_tf_config cfg{};
  Layout P;
  char* ws = nullptr;
  hipStream_t sf = nullptr, sb = nullptr;
  int device = 0;
  std::vector<hipEvent_t> ef;
  hipEvent_t ejoin = nullptr;
  erase_status sticky = ERASE_OK;
  std::string err;
  bool timing = false;
  std::vector<hipEvent_t> pool;
  size_t pool_used = 0;
  hipEvent_t t0 = nullptr, tn0 = nullptr, tn1 = nullptr;
  std::vector<Rec> recs, last;
  bool last_valid = false;
};

bool hip_ok(TfCtx* c, hipError_t e, const char* what) {
  if (e == hipSuccess) return true;
  char buf[256];
  std::snprintf(buf, sizeof buf, "%s: %s", what, hipGetErrorString(e));
  c->err = buf;
  c->sticky = ERASE_ERR_HIP;
  return false;
}
#define TFCHK(c, call)                                      \
  do {                                                      \
    if (!hip_ok((c), (call), #call)) return ERASE_ERR_HIP;  \
  } while (0)

// One launch, optionally timed with kernel-stamped events.
template <class F>
erase_status run(TfCtx* c, int kind, int b, int layer, int sid, double flops, double bytes, int grid, F&& fn,
                 int tm = 0, int tn = 0, int split = 0, bool stamped = true, hipStream_t s = nullptr) {
  LaunchEv ev;
  Rec rec{};
  if (c->timing) {
    if (c->pool_used + 2 > c->pool.size()) {
      c->err = "timing event pool exhausted";
      return ERASE_ERR_STATE;
    }
    rec.e0 = c->pool[c->pool_used++];
    rec.e1 = c->pool[c->pool_used++];
    if (stamped) {
      ev.e0 = rec.e0;
      ev.e1 = rec.e1;
    } else {
      TFCHK(c, hipEventRecord(rec.e0, s));
    }
  }
  if (!hip_ok(c, fn(ev), "kernel launch")) return ERASE_ERR_HIP;
  if (c->timing) {
    if (!stamped) TFCHK(c, hipEventRecord(rec.e1, s));
    rec.r.kind = kind;
    rec.r.block = b;
    rec.r.layer = layer;
    rec.r.stream = sid;
    rec.r.flops = flops;
    rec.r.bytes = bytes;
    rec.r.grid = grid;
    rec.r.tile_m = tm;
    rec.r.tile_n = tn;
    rec.r.split = split;
    c->recs.push_back(rec);
  }
  return ERASE_OK;
}
#define TFRUN(...)                                  \
  do {                                              \
    erase_status st_ = run(__VA_ARGS__);            \
    if (st_ != ERASE_OK) return st_;                \
  } while (0)

erase_status gemm(TfCtx* c, const Lin& L, int tkind, int b, int w, int sid, hipStream_t s) {
  const GemmDesc& g = L.g;
  const double flops = 2.0 * g.M * double(g.N) * g.K;
  const int grid = (int)(cdv(g.M, g.bm) * cdv(g.N, g.bn) * g.split);
  TFRUN(c, tkind, b, w, sid, flops, 0.0, grid, [&](const LaunchEv& ev) { return launch_gemm(1, L.kind, g, L.e, s, ev); },
        g.bm, g.bn, g.split);
  return ERASE_OK;
}

erase_status rms(TfCtx* c, int backward, const TfRmsArgs& a, int b, int layer, int sid, hipStream_t s) {
  const double bytes = double(a.N) * a.d * (backward ? (a.res ? 8 : 6) + (a.out_f32 ? 4 : 2) : 4);
  TFRUN(c, backward ? 13 : 12, b, layer, sid, 0.0, bytes, (int)cdv(a.N, 4),
        [&](const LaunchEv& ev) { return launch_tf_rms(backward, a, s, ev); });
  return ERASE_OK;
}

TfRmsArgs rms_args(const Layout& P, const uint16_t* x, float* r, uint16_t* y) {
  TfRmsArgs a{};
  a.x = x;
  a.ldx = P.ldd;
  a.y = y;
  a.ldy = P.ldd;
  a.r = r;
  a.N = P.D.N;
  a.d = P.D.d;
  a.eps = 1e-6f;
  return a;
}

TfAttnArgs attn_args(const Layout& P, const Block& B) {
  TfAttnArgs a{};
  a.qkv = B.qkv;
  a.ldqkv = P.ld3;
  a.o = B.o;
  a.ldo = P.ldd;
  a.lse = B.lse;
  a.dout = B.dout;
  a.lddo = P.ldd;
  a.dsum = B.dsum;
  a.dqkv = B.dqkv;
  a.lddqkv = P.ld3;
  a.B = P.D.B;
  a.T = P.D.T;
  a.H = P.D.H;
  a.d = P.D.d;
  a.scale = 0.125f;
  return a;
}

double attn_flops(const Dims& D) { return 2.0 * D.B * double(D.d) * D.T * (D.T + 1) / 2.0; }

// body forward of block b: embedding (block 0), attention, MLP
erase_status enqueue_body(TfCtx* c, int b, const int32_t* tokens, hipStream_t s, int sid) {
  const Layout& P = c->P;
  const Dims& D = P.D;
  const Block& B = P.blk[b];
  if (b == 0) {
    TfEmbedArgs e{};
    e.tokens = tokens;
    e.B = D.B;
    e.T = D.T;
    e.V = D.V;
    e.d = D.d;
    e.emb = B.cemb;
    e.ldemb = D.d;
    e.a0 = B.a0;
    e.lda0 = P.ldd;
    e.target = P.target;
    e.input = P.input;
    e.status = P.status;
    TFRUN(c, 11, b, -1, sid, 0.0, double(D.N) * (4.0 * D.d + 8.0), (int)cdv(D.N, 4),
          [&](const LaunchEv& ev) { return launch_tf_embed(e, s, ev); });
  }
  if (auto st = rms(c, 0, rms_args(P, B.a0, B.r1, B.n1), b, 0, sid, s); st != ERASE_OK) return st;
  if (auto st = gemm(c, B.fwd[WQKV], 1, b, WQKV, sid, s); st != ERASE_OK) return st;
  const TfAttnArgs at = attn_args(P, B);
  TFRUN(c, 14, b, 0, sid, 2.0 * attn_flops(D), 0.0, (int)(cdv(D.T, 64) * D.H * D.B),
        [&](const LaunchEv& ev) { return launch_tf_attn(0, at, s, ev); });
  if (auto st = gemm(c, B.fwd[WO], 1, b, WO, sid, s); st != ERASE_OK) return st;
  if (auto st = rms(c, 0, rms_args(P, B.a1, B.r2, B.n2), b, 1, sid, s); st != ERASE_OK) return st;
  if (auto st = gemm(c, B.fwd[W1], 1, b, W1, sid, s); st != ERASE_OK) return st;
  if (auto st = gemm(c, B.fwd[W2], 1, b, W2, sid, s); st != ERASE_OK) return st;
  return ERASE_OK;
}

// local head: norm (and the target logit), the logits GEMM storing the
// exponentials relative to the target logit with per-tile sums, then per row
// the loss and the scales of the head's gradient (Section 2.1: the block's
// own objective)
erase_status enqueue_head(TfCtx* c, int b, hipStream_t s, int sid) {
  const Layout& P = c->P;
  const Dims& D = P.D;
  const Block& B = P.blk[b];
  TfRmsArgs ra = rms_args(P, B.z, B.r3, B.hn);
  ra.hw = B.sh[WH];
  ra.ldhw = D.cols[WH];
  ra.target = P.target;
  ra.xref = B.xref;
  if (auto st = rms(c, 0, ra, b, 2, sid, s); st != ERASE_OK) return st;
  if (auto st = gemm(c, B.fwd[WH], 1, b, WH, sid, s); st != ERASE_OK) return st;
  TfHeadArgs x{};
  x.e = B.logits;
  x.lde = P.ldv;
  x.lstat = B.lstat;
  x.ldlstat = B.ntiles;
  x.ntiles = B.ntiles;
  x.xref = B.xref;
  x.target = P.target;
  x.hn = B.hn;
  x.ldhn = P.ldd;
  x.hns = B.hns;
  x.ldhns = P.ldd;
  x.w = B.sh[WH];
  x.ldw = D.cols[WH];
  x.rowscale = B.rowscale;
  x.rowloss = B.rowloss;
  x.flag = B.flag;
  x.N = D.N;
  x.V = D.V;
  x.d = D.d;
  x.scale = c->cfg.lambda / float(D.N);
  x.ploss = B.ploss;
  // bytes: per-tile sums, and the head input read and written scaled
  TFRUN(c, 16, b, 0, sid, 0.0, double(D.N) * (4.0 * B.ntiles + 4.0 * D.d + 16.0), (int)cdv(D.N, 4),
        [&](const LaunchEv& ev) { return launch_tf_head(0, x, s, ev); });
  TFRUN(c, 16, b, 1, sid, 0.0, double(D.N) * 4.0, (int)cdv(D.N, 4),
        [&](const LaunchEv& ev) { return launch_tf_head(1, x, s, ev); });
  return ERASE_OK;
}

erase_status enqueue_backward(TfCtx* c, int b, hipStream_t s, int sid) {
  Layout& P = c->P;
  const Dims& D = P.D;
  const Block& B = P.blk[b];
  auto G = [&](const Lin& L, int tk, int w) { return gemm(c, L, tk, b, w, sid, s); };
  // both gradient GEMMs of weight w (one launch when grouped)
  auto G2 = [&](int w) {
    if (!B.grouped[w]) {
      erase_status e2 = G(B.dgr[w], 4, w);
      return e2 != ERASE_OK ? e2 : G(B.wgr[w], 3, w);
    }
    const GemmDesc &gd = B.dgr[w].g, &gw = B.wgr[w].g;
    const double flops = 2.0 * gd.M * double(gd.N) * gd.K + 2.0 * gw.M * double(gw.N) * gw.K;
    const int grid = (int)(cdv(gd.M, gd.bm) * cdv(gd.N, gd.bn) + cdv(gw.M, gw.bm) * cdv(gw.N, gw.bn) * gw.split);
    return run(c, 6, b, w, sid, flops, 0.0, grid,
               [&](const LaunchEv& ev) { return launch_bwd_gemm(1, gd, B.dgr[w].e, gw, B.wgr[w].e, s, ev); },
               gd.bm, gd.bn, gw.split);
  };
  erase_status st;
  if ((st = G2(WH)) != ERASE_OK) return st;
  {  // dz = rms'(z) (rowscale dhn): the head's input gradient takes its row scale here
    TfRmsArgs a = rms_args(P, B.z, B.r3, B.dz);
    a.dy = B.dhn;
    a.lddy = P.ldd;
    a.dyscale = B.rowscale;
    if ((st = rms(c, 1, a, b, 2, sid, s)) != ERASE_OK) return st;
  }
  if ((st = G(B.dgr[W2], 4, W2)) != ERASE_OK) return st;
  if ((st = G(B.wgr[W2], 3, W2)) != ERASE_OK) return st;
  if ((st = G2(W1)) != ERASE_OK) return st;
  {  // da1 = dz + rms'(a1) dn2
    TfRmsArgs a = rms_args(P, B.a1, B.r2, B.da1);
    a.dy = B.dn2;
    a.lddy = P.ldd;
    a.res = B.dz;
    a.ldres = P.ldd;
    if ((st = rms(c, 1, a, b, 1, sid, s)) != ERASE_OK) return st;
  }
  if ((st = G2(WO)) != ERASE_OK) return st;
  const TfAttnArgs at = attn_args(P, B);
  const int ga = (int)(cdv(D.T, 64) * D.H * D.B);
  TFRUN(c, 15, b, 1, sid, 0.0, double(D.N) * D.d * 4.0, (int)cdv(int64_t(D.N) * D.H, 32),
        [&](const LaunchEv& ev) { return launch_tf_attn(1, at, s, ev); });
  TFRUN(c, 15, b, 2, sid, 4.0 * attn_flops(D), 0.0, ga, [&](const LaunchEv& ev) { return launch_tf_attn(2, at, s, ev); });
  TFRUN(c, 15, b, 3, sid, 3.0 * attn_flops(D), 0.0, ga, [&](const LaunchEv& ev) { return launch_tf_attn(3, at, s, ev); });
  if (b == 0) {
    if ((st = G2(WQKV)) != ERASE_OK) return st;
    TfRmsArgs a = rms_args(P, B.a0, B.r1, nullptr);
    a.dy = B.dn1;
    a.lddy = P.ldd;
    a.res = B.da1;
    a.ldres = P.ldd;
    a.out_f32 = B.da0;
    a.ldout = P.ldd;
    if ((st = rms(c, 1, a, b, 0, sid, s)) != ERASE_OK) return st;
    TfEmbGradArgs e{};
    e.input = P.input;
    e.N = D.N;
    e.V = D.V;
    e.d = D.d;
    e.count = P.count;
    e.start = P.start;
    e.fill = P.fill;
    e.bucket = P.bucket;
    e.dx = B.da0;
    e.lddx = P.ldd;
    e.grad = B.gemb;
    e.ldgrad = D.d;
    TFRUN(c, 17, b, -1, sid, 0.0, double(D.N) * D.d * 4.0 + double(D.V) * D.d * 4.0, (int)cdv(D.V, 4),
          [&](const LaunchEv&) { return launch_tf_emb_grad(e, s); }, 0, 0, 0, false, s);
  } else if ((st = G(B.wgr[WQKV], 3, WQKV)) != ERASE_OK) {
    return st;
  }
  return ERASE_OK;
}

erase_status enqueue_adam(TfCtx* c, int b, float* losses, hipStream_t s, int sid) {
  const Layout& P = c->P;
  const Block& B = P.blk[b];
  AdamArgs a{};
  a.seg = B.segs_dev;
  a.nseg = (int)B.segs.size();
  for (int i = 0; i < a.nseg; ++i) a.chunk0[i] = B.segs[i].chunk0;
  a.nchunks = B.nchunks;
  a.hyper = P.hyper;
  a.beta1 = c->cfg.beta1;
  a.beta2 = c->cfg.beta2;
  a.eps = c->cfg.eps;
  a.ploss = B.ploss;
  a.nloss = B.nloss;
  a.inv_m = 1.0f / float(P.D.N);
  a.loss_out = losses + b;
  a.status = P.status;
  double bytes = 0;
  for (const AdamSeg& sg : B.segs)
    bytes += double(sg.rows) * sg.cols * (4.0 * sg.nsplit + 24.0 + (sg.g ? 4.0 : 0.0) + (sg.sh ? 2 : 0) + (sg.sht ? 2 : 0));
  TFRUN(c, 5, b, -1, sid, 0.0, bytes, (int)B.nchunks, [&](const LaunchEv& ev) { return launch_adam(1, a, s, ev); });
  return ERASE_OK;
}

erase_status enqueue_step(TfCtx* c, const int32_t* tokens, int sched, float* losses) {
  Layout& P = c->P;
  const int L = P.D.L;
  PrologueArgs pa{};
  pa.t = P.t;
  pa.hyper = P.hyper;
  pa.lr = c->cfg.lr;
  pa.beta1 = c->cfg.beta1;
  pa.beta2 = c->cfg.beta2;
  TFRUN(c, 0, -1, -1, 0, 0.0, 16.0, 1, [&](const LaunchEv& ev) { return launch_prologue(1, pa, c->sf, ev); });
  erase_status st;
  if (sched == ERASE_SCHED_SERIAL) {
    for (int b = 0; b < L; ++b) {
      if ((st = enqueue_body(c, b, tokens, c->sf, 0)) != ERASE_OK) return st;
      if ((st = enqueue_head(c, b, c->sf, 0)) != ERASE_OK) return st;
    }
    for (int b = L - 1; b >= 0; --b)
      if ((st = enqueue_backward(c, b, c->sf, 0)) != ERASE_OK) return st;
    for (int b = 0; b < L; ++b)
      if ((st = enqueue_adam(c, b, losses, c->sf, 0)) != ERASE_OK) return st;
    return ERASE_OK;
  }
  // OVERLAP
  for (int b = 0; b < L; ++b) {
    if ((st = enqueue_body(c, b, tokens, c->sf, 0)) != ERASE_OK) return st;
    TFCHK(c, hipEventRecord(c->ef[b], c->sf));
    TFCHK(c, hipStreamWaitEvent(c->sb, c->ef[b], 0));
    if ((st = enqueue_head(c, b, c->sb, 1)) != ERASE_OK) return st;
    if ((st = enqueue_backward(c, b, c->sb, 1)) != ERASE_OK) return st;
    if ((st = enqueue_adam(c, b, losses, c->sb, 1)) != ERASE_OK) return st;
  }
  TFCHK(c, hipEventRecord(c->ejoin, c->sb));
  TFCHK(c, hipStreamWaitEvent(c->sf, c->ejoin, 0));
  return ERASE_OK;
}

erase_status refresh(TfCtx* c) {
  for (const Block& B : c->P.blk) {
    AdamArgs a{};
    a.seg = B.segs_dev;
    a.nseg = (int)B.segs.size();
    for (int i = 0; i < a.nseg; ++i) a.chunk0[i] = B.segs[i].chunk0;
    a.nchunks = B.nchunks;
    TFCHK(c, launch_refresh(1, a, c->sf));
  }
  return ERASE_OK;
}

}  // namespace

// The opaque context handle of the C ABI.
struct erase_tf_ctx {
  TfCtx impl;
};

namespace {
TfCtx* as_ctx(erase_tf_ctx* p) { return p ? &p->impl : nullptr; }
}  // namespace

extern "C" {

erase_status erase_tf_param_count(const erase_tf_config* cfg, int32_t block, int64_t* count) {
  if (!count) return ERASE_ERR_INVALID_ARG;
  if (erase_status st = validate(cfg, nullptr); st != ERASE_OK) return st;
  if (block < 0 || block >= cfg->n_layers) return ERASE_ERR_INVALID_ARG;
  *count = param_count(dims_of(*cfg), block);
  return ERASE_OK;
}

erase_status erase_tf_workspace_bytes(const erase_tf_config* cfg, size_t* bytes) {
  if (!bytes) return ERASE_ERR_INVALID_ARG;
  if (erase_status st = validate(cfg, nullptr); st != ERASE_OK) return st;
  Layout P;
  *bytes = build_layout(*cfg, 0, &P);
  return ERASE_OK;
}

erase_status erase_tf_init(const erase_tf_config* cfg, const erase_block_buffers* bufs, void* workspace,
                           size_t ws_bytes, void* s_fwd, void* s_bwd, erase_tf_ctx** ctx_out) {
  if (!ctx_out) return ERASE_ERR_INVALID_ARG;
  *ctx_out = nullptr;
  if (erase_status st = validate(cfg, nullptr); st != ERASE_OK) return st;
  if (!bufs) return ERASE_ERR_INVALID_ARG;
  for (int b = 0; b < cfg->n_layers; ++b) {
    if (!bufs[b].param || !bufs[b].m || !bufs[b].v) return ERASE_ERR_INVALID_ARG;
    const uintptr_t al = reinterpret_cast<uintptr_t>(bufs[b].param) | reinterpret_cast<uintptr_t>(bufs[b].m) |
                         reinterpret_cast<uintptr_t>(bufs[b].v) | reinterpret_cast<uintptr_t>(bufs[b].grad);
    if (al % 4) return ERASE_ERR_INVALID_ARG;
  }
  if (!s_fwd || !s_bwd || s_fwd == s_bwd) return ERASE_ERR_INVALID_ARG;
  if (!workspace || reinterpret_cast<uintptr_t>(workspace) % kAlign) return ERASE_ERR_WORKSPACE;
  {
    Layout probe;
    if (ws_bytes < build_layout(*cfg, 0, &probe)) return ERASE_ERR_WORKSPACE;
  }
  erase_tf_ctx* h = new erase_tf_ctx();
  TfCtx* c = &h->impl;
  c->cfg = *cfg;
  c->ws = static_cast<char*>(workspace);
  c->sf = static_cast<hipStream_t>(s_fwd);
  c->sb = static_cast<hipStream_t>(s_bwd);
  build_layout(c->cfg, reinterpret_cast<uintptr_t>(workspace), &c->P);
  build_gemms(c->cfg, &c->P);
  build_segments(&c->P, bufs);
  auto bail = [&](erase_status s) {
    for (hipEvent_t e : c->ef) (void)hipEventDestroy(e);
    if (c->ejoin) (void)hipEventDestroy(c->ejoin);
    delete h;
    return s;
  };
  if (hipGetDevice(&c->device) != hipSuccess) return bail(ERASE_ERR_HIP);
  // ordering events between this device's streams only (no host waits on
  // them): recorded without the system-scope fence
  const unsigned evflags = hipEventDisableTiming | hipEventDisableSystemFence;
  for (int b = 0; b < cfg->n_layers; ++b) {
    hipEvent_t e;
    if (hipEventCreateWithFlags(&e, evflags) != hipSuccess) return bail(ERASE_ERR_HIP);
    c->ef.push_back(e);
  }
  if (hipEventCreateWithFlags(&c->ejoin, evflags) != hipSuccess) return bail(ERASE_ERR_HIP);
  // zero the workspace once: counters, and the padding rows and columns every
  // GEMM operand relies on (nothing writes outside the logical extents)
  if (hipMemsetAsync(c->ws, 0, c->P.bytes, c->sf) != hipSuccess) return bail(ERASE_ERR_HIP);
  for (Block& B : c->P.blk)
    if (hipMemcpyAsync(B.segs_dev, B.segs.data(), sizeof(AdamSeg) * B.segs.size(), hipMemcpyHostToDevice, c->sf) !=
        hipSuccess)
      return bail(ERASE_ERR_HIP);
  if (refresh(c) != ERASE_OK) return bail(ERASE_ERR_HIP);
  *ctx_out = h;
  return ERASE_OK;
}

erase_status erase_tf_step(erase_tf_ctx* ctx, const int32_t* tokens, int32_t schedule, float* losses) {
  TfCtx* c = as_ctx(ctx);
  if (!c || !tokens || !losses) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (reinterpret_cast<uintptr_t>(tokens) % 4 || reinterpret_cast<uintptr_t>(losses) % 4) return ERASE_ERR_INVALID_ARG;
  if (schedule != ERASE_SCHED_SERIAL && schedule != ERASE_SCHED_OVERLAP) return ERASE_ERR_UNSUPPORTED;
  int dev = -1;
  TFCHK(c, hipGetDevice(&dev));
  if (dev != c->device) {
    c->err = "current device differs from the context's";
    return ERASE_ERR_INVALID_ARG;
  }
  c->recs.clear();
  c->pool_used = 0;
  if (c->timing) {
    TFCHK(c, hipEventRecord(c->t0, c->sf));
    TFCHK(c, hipEventRecord(c->tn0, c->sf));
    TFCHK(c, hipEventRecord(c->tn1, c->sf));
  }
  erase_status st = enqueue_step(c, tokens, schedule, losses);
  if (st != ERASE_OK) {
    if (c->sticky == ERASE_OK) c->sticky = st;
    return st;
  }
  if (c->timing) {
    c->last = c->recs;
    c->last_valid = true;
  }
  return ERASE_OK;
}

erase_status erase_tf_sync(erase_tf_ctx* ctx) {
  TfCtx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  TFCHK(c, hipStreamSynchronize(c->sf));
  TFCHK(c, hipStreamSynchronize(c->sb));
  int status = 0;
  TFCHK(c, hipMemcpy(&status, c->P.status, sizeof(int), hipMemcpyDeviceToHost));
  if (status == 2) {
    c->sticky = ERASE_ERR_INVALID_ARG;
    c->err = "a token id was outside [0, vocab)";
    return ERASE_ERR_INVALID_ARG;
  }
  if (status != 0) {
    c->sticky = ERASE_ERR_NONFINITE;
    c->err = "a block loss was not finite";
    return ERASE_ERR_NONFINITE;
  }
  return ERASE_OK;
}

erase_status erase_tf_get_step(erase_tf_ctx* ctx, int64_t* t) {
  TfCtx* c = as_ctx(ctx);
  if (!c || !t) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  TFCHK(c, hipStreamSynchronize(c->sb));
  TFCHK(c, hipMemcpyAsync(t, c->P.t, sizeof(int64_t), hipMemcpyDeviceToHost, c->sf));
  TFCHK(c, hipStreamSynchronize(c->sf));
  return ERASE_OK;
}

erase_status erase_tf_set_step(erase_tf_ctx* ctx, int64_t t) {
  TfCtx* c = as_ctx(ctx);
  if (!c || t < 0) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  TFCHK(c, hipStreamSynchronize(c->sb));
  TFCHK(c, hipMemcpyAsync(c->P.t, &t, sizeof(int64_t), hipMemcpyHostToDevice, c->sf));
  TFCHK(c, hipStreamSynchronize(c->sf));
  return ERASE_OK;
}

erase_status erase_tf_refresh_weights(erase_tf_ctx* ctx) {
  TfCtx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  TFCHK(c, hipStreamSynchronize(c->sb));
  return refresh(c);
}

erase_status erase_tf_set_timing(erase_tf_ctx* ctx, int32_t enable) {
  TfCtx* c = as_ctx(ctx);
  if (!c) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (enable && c->pool.empty()) {
    const size_t need = size_t(2) * (40 * c->P.D.L + 16);
    for (size_t i = 0; i < need; ++i) {
      hipEvent_t e;
      TFCHK(c, hipEventCreate(&e));
      c->pool.push_back(e);
    }
    TFCHK(c, hipEventCreate(&c->t0));
    TFCHK(c, hipEventCreate(&c->tn0));
    TFCHK(c, hipEventCreate(&c->tn1));
  }
  c->timing = enable != 0;
  c->last_valid = false;
  return ERASE_OK;
}

erase_status erase_tf_read_timing(erase_tf_ctx* ctx, erase_kernel_time* out, int32_t cap, int32_t* n) {
  TfCtx* c = as_ctx(ctx);
  if (!c || !n || cap < 0 || (cap > 0 && !out)) return ERASE_ERR_INVALID_ARG;
  if (c->sticky != ERASE_OK) return ERASE_ERR_STATE;
  if (!c->last_valid) return ERASE_ERR_STATE;
  *n = (int32_t)(c->last.size() + 1);
  auto ms = [&](hipEvent_t e, float* v) { return hipEventElapsedTime(v, c->t0, e); };
  if (cap > 0) {
    erase_kernel_time r0{};
    r0.kind = 7;
    r0.block = -1;
    r0.layer = -1;
    TFCHK(c, ms(c->tn0, &r0.start_ms));
    TFCHK(c, ms(c->tn1, &r0.end_ms));
    out[0] = r0;
  }
  for (size_t i = 0; i < c->last.size() && int32_t(i + 1) < cap; ++i) {
    erase_kernel_time r = c->last[i].r;
    TFCHK(c, ms(c->last[i].e0, &r.start_ms));
    TFCHK(c, ms(c->last[i].e1, &r.end_ms));
    out[i + 1] = r;
  }
  return ERASE_OK;
}

erase_status erase_tf_tensor(erase_tf_ctx* ctx, int32_t block, int32_t which, void** ptr, int64_t* ld) {
  TfCtx* c = as_ctx(ctx);
  if (!c || !ptr || !ld || block < 0 || block >= c->P.D.L) return ERASE_ERR_INVALID_ARG;
  const Layout& P = c->P;
  const Block& B = P.blk[block];
  void* p = nullptr;
  int64_t l = P.ldd;
  switch (which) {
    case 0: p = B.a0; break;
    case 1: p = B.n1; break;
    case 2: p = B.qkv; l = P.ld3; break;
    case 3: p = B.o; break;
    case 4: p = B.a1; break;
    case 5: p = B.n2; break;
    case 6: p = B.u; l = P.ld4; break;
    case 7: p = B.g; l = P.ld4; break;
    case 8: p = B.z; break;
    case 9: p = B.hn; break;
    case 10: p = B.logits; l = P.ldv; break;
    case 11: p = B.lse; l = P.D.T; break;
    case 12: p = B.dqkv; l = P.ld3; break;
    case 13: p = B.dz; break;
    case 14: p = B.rowscale; l = P.D.N; break;
    case 15: p = B.hns; break;
    default: return ERASE_ERR_INVALID_ARG;
  }
  *ptr = p;
  *ld = l;
  return ERASE_OK;
}

erase_status erase_tf_destroy(erase_tf_ctx* ctx) {
  TfCtx* c = as_ctx(ctx);
  if (!c) return ERASE_OK;
  (void)hipStreamSynchronize(c->sf);
  (void)hipStreamSynchronize(c->sb);
  for (hipEvent_t e : c->ef) (void)hipEventDestroy(e);
  if (c->ejoin) (void)hipEventDestroy(c->ejoin);
  for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
  for (hipEvent_t e : {c->t0, c->tn0, c->tn1})
    if (e) (void)hipEventDestroy(e);
  delete ctx;
  return ERASE_OK;
}

const char* erase_tf_last_error(erase_tf_ctx* ctx) {
  TfCtx* c = as_ctx(ctx);
  return c ? c->err.c_str() : "";
}

}  // extern "C"
