// Internal interface between the dispatcher (erase_api.cpp) and the HIP
// kernels (kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace erase {

// One GEMM launch, fp32 accumulation:
//   forward / input gradient: C[m][n] = sum_k A[m][k] * B[n][k] (both
//     operands stored with the contraction index contiguous);
//   weight gradient (GK_WGRAD): C[m][n] = sum_k A[k][m] * B[k][n] (both
//     operands row-major over the contraction: activation gradient and layer
//     input as produced).
// The contraction range is split into `split` slices of `kps` elements.
//
// Operand contract (no loads are masked): K is the padded contraction length,
// a multiple of the k-step (64 bf16 / 32 fp32 elements).  Forward / input
// gradient: A holds at least roundup(M, 128) rows and B roundup(N, 128) rows
// of at least K elements.  Weight gradient: A and B hold at least K rows of
// at least roundup(M, 128) and roundup(N, 128) elements.  Every element
// outside the logical block is zero.  M and N are the logical output extents
// the epilogue stores.
struct GemmDesc {
  const void* A;
  int64_t lda;
  const void* B;
  int64_t ldb;
  int M, N, K;
  int kps;
  int split;
  int bm, bn;  // workgroup tile
  int group;   // M-tiles per group of the XCD-aware tile order (0: launcher picks)
  int kgroups; // 2: two k-groups of four waves (bf16 64x128 / 64x64 forward tiles); else one
};

// M-tiles per group of the XCD-aware tile order (see tile_from in the
// kernels): the group size that minimises the A and B rows one XCD's
// contiguous range of tiles touches.
int xcd_group(int gm, int gn, int split, int bm, int bn);

// GK_FWD_HEAD: the last linear+ReLU layer of a block with the local head
// (Section 2.1) fused into its epilogue; the tile spans the whole width
// (N <= BN), so each workgroup holds complete rows of the block output.
//
// Transformer kinds (bf16 only):
//   GK_FWD_LIN     y = acc (+ res)                       (projections, residual adds)
//   GK_FWD_GELU    y = gelu(acc), and acc itself into gout (the MLP up-projection)
//   GK_DGRAD_GELU  g = acc * gelu'(u), u read from mask  (input gradient below the GELU)
//   GK_FWD_LOGITS  y = exp(acc - xref[m]) (the row's exponentials relative to a
//                  reference logit), plus per row the sum of the stored values
//                  over this tile's columns into lstat    (vocabulary head)
// GK_DGRAD with neither mask nor below_cross stores g = acc (+ res) as is.
enum GemmKind {
  GK_FWD_RELU = 0, GK_FWD_CROSS = 1, GK_WGRAD = 2, GK_DGRAD = 3, GK_FWD_HEAD = 4,
  GK_FWD_LIN = 5, GK_FWD_GELU = 6, GK_DGRAD_GELU = 7, GK_FWD_LOGITS = 8
};

// Optional events of one launch: when either is set, the kernel is dispatched
// with hipExtLaunchKernelGGL, which stamps e0/e1 at the kernel's own start
// and end on the device (timing: both; e1 alone: a stream-ordering event
// recorded by the launch itself, with no packet of its own).
struct LaunchEv {
  hipEvent_t e0 = nullptr, e1 = nullptr;
};

// Epilogue operands.  Which fields are read depends on the GemmKind.
struct EpiParams {
  // forward: y = relu(acc + bias) or x0 * (acc + bias) + xl
  const float* bias;
  void* y;   int64_t ldy;    // [M][ldy] row-major output
  const void* x0; int64_t ldx0;  // block input (cross forward, and cross-below dgrad)
  const void* xl; int64_t ldxl;  // layer input (cross forward residual)
  // weight gradient: part[z][m][n], row sums of A into bpart[z][m]
  float* part; int64_t ldp; int64_t pstride;
  float* bpart;
  // input gradient: g = acc (+ res); below relu: g*[mask>0]; below cross: g, g*x0
  const void* res;  int64_t ldres;
  const void* mask; int64_t ldmask;
  void* gout; int64_t ldgout;
  void* dmn;  int64_t lddmn;
  int below_cross;
  // fused head: s = z hw + hc, loss and ds = lam (sigmoid(s) - y) inv_m,
  // dz = ds hw [z > 0] into dmn, per-M-tile partials
  const float* hw;
  const float* hc;
  const float* labels;
  float lam, inv_m;
  float* pdw;    // [M-tiles][N]
  float* pdc;    // [M-tiles]
  float* ploss;  // [M-tiles]
  // weight gradient with the Adam update fused (ap non-null; unsplit
  // contraction): the workgroup updates its tile of the parameter matrix
  // [M][N] (flat, row-major), its Adam state, the gradient (ag nullable) and
  // the GEMM copy [M][ldash] from the finished gradient tile; no partial
  // slice is stored
  float* ap; float* am; float* av; float* ag;
  void* ash; int64_t ldash;
  const float* hyper;  // lr / (1 - beta1^t), sqrt(1 - beta2^t) of this step
  float b1, b2, eps;
  // and the bias's Adam update from the tiles' row sums of the A operand
  // (bp non-null: the tiles of the first column block update bias entries
  // [0, M), and no row sum is stored in bpart); gradient bg nullable
  float* bp; float* bm; float* bv; float* bg;
  // logits (GK_FWD_LOGITS): lstat[m][t] = sum over the columns of N-tile t
  // of the stored (bf16) values exp(acc - xref[m]) of row m
  float* lstat; int64_t ldlstat;
  const float* xref;
};

hipError_t launch_gemm(int bf16, int kind, const GemmDesc& g, const EpiParams& e, hipStream_t s,
                       const LaunchEv& ev = {});
// Input-gradient (gd, split 1) and weight-gradient (gw) GEMMs of one layer in
// one launch; both must use the same tile, 64x64 or 128x128.
hipError_t launch_bwd_gemm(int bf16, const GemmDesc& gd, const EpiParams& ed, const GemmDesc& gw, const EpiParams& ew,
                           hipStream_t s, const LaunchEv& ev = {});

// Step prologue: t += 1 and the zero-padded copy xp[m][k] = x[m][k] (its
// padding stays zero).
// Workspace header (first 256 bytes): step counter t (int64 at 0), status
// word (int32 at 8), and the Adam step factors written by the prologue, one
// pair per step parity p: lr / (1 - beta1^t) (float at 16 + 8p) and
// sqrt(1 - beta2^t) (float at 20 + 8p).
struct PrologueArgs {
  int64_t* t;
  float* hyper;  // this step's Adam factors (one pair per step parity)
  float lr, beta1, beta2;
  const void* x; int64_t ldx;
  void* xp; int64_t ldxp;
  int M, K;
};
hipError_t launch_prologue(int bf16, const PrologueArgs& a, hipStream_t s, const LaunchEv& ev = {});

// Fused local head + sigmoid-BCE + gradient at z (one workgroup per 64 rows).
struct HeadArgs {
  const void* z; int64_t ldz;    // [M][N] block output
  const float* w;                // head weight [N] (fp32 master)
  const float* c;                // head bias [1]
  const float* y;                // labels [M]
  float lam, inv_m;
  int M, N;
  void* dmn; int64_t lddmn;      // dz row-major
  float* pdw;                    // [nblk][N]
  float* pdc;                    // [nblk]
  float* ploss;                  // [nblk]
};
// Rows of z per head workgroup: the [rows][N] tile is staged in LDS (at most
// 64 KiB), 32 rows when it fits, never fewer than one 16-byte column item.
constexpr int HEAD_MAX_N = 2048;
__host__ __device__ inline int head_pitch(int N, int esz) {  // elements per LDS row: 16-byte multiple plus one chunk
  const int kch = 16 / esz;
  return (N + kch - 1) / kch * kch + kch;
}
__host__ __device__ inline int head_rows(int N, int esz) {
  int r = 32;
  while (r > 16 / esz && r * head_pitch(N, esz) * esz > 65536) r /= 2;
  return r;
}
inline size_t head_lds_bytes(int N, int esz) { return (size_t)head_rows(N, esz) * head_pitch(N, esz) * esz; }
hipError_t launch_head(int bf16, const HeadArgs& a, hipStream_t s, const LaunchEv& ev = {});

// Fused split-reduction + Adam + GEMM-copy refresh for one block.  The
// segment table lives in device memory (written once at init).  A segment
// is a [rows][cols] parameter matrix (a vector is one row) processed in
// tiles of ADAM_TR rows x ADAM_TC columns, one workgroup per tile (a
// thread owns 4 columns of one row of a matrix tile, one element of a
// vector).
constexpr int ADAM_TR = 16, ADAM_TC = 64;
struct AdamSeg {
  float* p; float* m; float* v; float* g;   // flat [rows*cols] fp32 (g nullable)
  const float* part;                        // partial sums [nsplit][rows][ldpart]
  int64_t pstride;
  int rows, cols, ldpart, nsplit;
  void* sh;  int64_t ldsh;                  // GEMM copy [rows][ldsh], nullable
  void* sht; int64_t ldsht;                 // transposed GEMM copy [cols][ldsht], nullable
  int64_t chunk0;                           // first tile index of this segment
  int tcols;                                // tiles per row of tiles: ceil(cols / ADAM_TC)
};
constexpr int ADAM_MAX_SEG = 34;  // 16 layers x (W, b) + head (w, c)
struct AdamArgs {
  const AdamSeg* seg;  // device [nseg]
  int64_t chunk0[ADAM_MAX_SEG];  // first chunk of each segment (kernel-argument copy)
  int nseg;
  int64_t nchunks;
  const float* hyper;  // [step factor, sqrt bias correction 2] of this step (workspace header)
  float beta1, beta2, eps;
  const float* ploss; int nloss; float inv_m;  // loss finalize (nullable ploss)
  float* loss_out;
  int* status;
};
hipError_t launch_adam(int bf16, const AdamArgs& a, hipStream_t s, const LaunchEv& ev = {});

// A block's first-layer weight gradient with its fused Adam (g: 64x64, two
// k-groups, unsplit; e.ap set) and the Adam launch `a` of the block's other
// parameters in one launch (extra workgroups beside the GEMM tiles).
hipError_t launch_wgrad_adam(int bf16, const GemmDesc& g, const EpiParams& e, const AdamArgs& a, hipStream_t s,
                             const LaunchEv& ev = {});

// Weight copies only (init / refresh): same segments, no update.
hipError_t launch_refresh(int bf16, const AdamArgs& a, hipStream_t s);

// Embedding-bag input stage: x[m] = [log1p(dense[m]) | bag sums | 0...].
// Bag m of table t is indices[offsets[t][m] .. offsets[t][m+1]); rows of
// table t are tables[t][row][0 .. dim).  Invalid offsets or indices are
// skipped (read nothing) and set status[0] = 1 (status nullable).
struct EmbedArgs {
  const float* dense;     // [M][n_dense]
  const int64_t* offsets; // [T][M+1]
  const int32_t* indices; // [nnz]
  const float* tables;    // [T][rows][dim], 16-byte aligned
  void* x; int64_t ldx;   // [M][ldx] of the activation dtype
  int* status;
  int64_t nnz, rows;
  int M, n_dense, T, dim;  // dim % 4 == 0, 4 <= dim <= 256
};
hipError_t launch_embed_bags(int bf16, const EmbedArgs& a, hipStream_t s);

// Backward of the embedding-bag stage: grad[t][r][d] = sum over the entries
// i of table t's bags with indices[i] == r of dx[bag m][n_dense + t dim + d],
// entries in increasing order; rows no entry selects are zero.  Bags must
// not overlap.  Scratch (all int32): count, start, fill [trows], bucket,
// gid, owner, bagm [nnz], large [nnz / 65 + 1], nlarge [1], bsum [trows / 4096 + 1].
// Invalid offsets or ids set status[0] = 1 (nullable).
struct EmbedBwdArgs {
  const int64_t* offsets;  // [T][M+1]
  const int32_t* indices;  // [nnz]
  const void* dx; int64_t lddx;  // [M][lddx] of the activation dtype
  float* grad;             // [T][rows][dim]
  int32_t* count; int32_t* start; int32_t* bucket; int32_t* gid; int32_t* owner; int32_t* slot;
  int32_t* large; int32_t* small; int32_t* nlarge; int32_t* bsum; int32_t* bsum2;
  int* status;
  int64_t nnz, trows;      // trows = T * rows < 2^31
  int rows, M, n_dense, T, dim;
};
hipError_t launch_embed_bags_backward(int bf16, const EmbedBwdArgs& a, hipStream_t s);
// Device address, on the current device, of the library's static scratch of
// the allocation-free backward (bytes: its size); looked up once per device.
hipError_t bag_scratch_device_ptr(void** ptr, size_t* bytes);

// ---------------------------------------------------------------------------
// small-transformer kernels (transformer.hip), bf16 activations
// ---------------------------------------------------------------------------
// a0[n] = emb[tokens[b][t]] (n = b T + t), input[n] = that token,
// target[n] = tokens[b][t + 1]; an id outside [0, V) reads nothing (zero row,
// id -1) and sets status[0] = 2.
struct TfEmbedArgs {
  const int32_t* tokens;  // [B][T + 1]
  int B, T, V, d;
  const uint16_t* emb; int64_t ldemb;  // bf16 copy [V][ldemb]
  uint16_t* a0; int64_t lda0;
  int32_t* target;
  int32_t* input;
  int* status;
};
hipError_t launch_tf_embed(const TfEmbedArgs& a, hipStream_t s, const LaunchEv& ev = {});

// Forward: y = x r, r = 1 / sqrt(mean(x^2) + eps) per row (r written); with
// hw set (the vocabulary head's bf16 weight [V][ldhw]), also the target
// logit xref[n] = y[n] . hw[target[n]] of the stored row (0 where the target
// is invalid).
// Backward: dx = r (s dy - y mean(s dy y)) + res (res nullable), y = x r,
// s = dyscale[n] (1 when dyscale is null), into out_f32 (fp32) when set,
// else y (bf16).  N rows of width d (d % 8 == 0, d <= 4096).
struct TfRmsArgs {
  const uint16_t* x; int64_t ldx;
  uint16_t* y; int64_t ldy;
  float* r;
  const uint16_t* dy; int64_t lddy;
  const float* dyscale;
  const uint16_t* res; int64_t ldres;
  float* out_f32; int64_t ldout;
  const uint16_t* hw; int64_t ldhw;
  const int32_t* target;
  float* xref;
  int64_t N;
  int d;
  float eps;
};
hipError_t launch_tf_rms(int backward, const TfRmsArgs& a, hipStream_t s, const LaunchEv& ev = {});

// Causal attention over qkv [B T][3 d] (q | k | v, head h at columns
// 64 h .. 64 h + 63 of each), head size 64.  part 0: o and lse
// [B][H][T] (natural log); 1: dsum = rowsum(dout * o); 2: dK and dV; 3: dQ,
// into dqkv (same layout as qkv).
struct TfAttnArgs {
  const uint16_t* qkv; int64_t ldqkv;
  uint16_t* o; int64_t ldo;
  float* lse;
  const uint16_t* dout; int64_t lddo;
  float* dsum;
  uint16_t* dqkv; int64_t lddqkv;
  int B, T, H, d;
  float scale;  // 1 / sqrt(64)
};
hipError_t launch_tf_attn(int part, const TfAttnArgs& a, hipStream_t s, const LaunchEv& ev = {});

// Softmax cross-entropy of the vocabulary head without a pass over the
// logits.  The logits GEMM stores e[n][v] = exp(x[n][v] - xref[n]) (bf16),
// xref[n] the target logit, and per-tile sums of e.  With S_n = sum_v e[n][v]
// the loss is lse - x_target = log S_n and the logit gradient is
// scale (e / S_n - onehot) = (scale / S_n) (e - S_n onehot).  So the head's
// gradient GEMMs take e with its target entry replaced by e - S_n as the
// output gradient, the input gradient is scaled per row afterwards
// (rowscale[n] = scale / S_n, applied by the RMSNorm backward), and the
// weight gradient takes hns[n] = rowscale[n] hn[n] as its second operand.
//   part 0 (one wave per row, four rows per workgroup): S_n from lstat, the
//     loss, rowscale, the target entry, hns; a row whose S_n falls outside
//     [2^-60, 2^60] (exponentials relative to the target logit out of range)
//     is flagged instead;
//   part 1 (one workgroup per four rows): every flagged row recomputed from
//     hn and w with the row's exact maximum as the reference, then the same
//     outputs; flags cleared.  Nothing to do for a row that is not flagged.
// ploss[g] = sum of the losses of rows 4 g .. 4 g + 3 (rowloss keeps each).
// flag [N] must be zero on entry to part 0 (part 1 leaves it zero).
struct TfHeadArgs {
  uint16_t* e; int64_t lde;         // [N][lde] exponentials (bf16), in place
  const float* lstat; int64_t ldlstat;
  int ntiles;
  const float* xref;
  const int32_t* target;
  const uint16_t* hn; int64_t ldhn;  // head input (bf16)
  uint16_t* hns; int64_t ldhns;      // scaled head input (bf16)
  const uint16_t* w; int64_t ldw;    // head weight [V][ldw] (bf16)
  float* rowscale;
  float* rowloss;
  int32_t* flag;
  int64_t N;
  int V, d;
  float scale;  // lam / N
  float* ploss;
};
hipError_t launch_tf_head(int part, const TfHeadArgs& a, hipStream_t s, const LaunchEv& ev = {});

// Embedding gradient: grad[v] = sum over positions n with input[n] == v, in
// increasing n, of dx[n] (fp32); zero rows for absent tokens.  count and
// fill [V] must be zero on entry (count is zero again on exit); start [V],
// bucket [N] scratch.  Four launches.
struct TfEmbGradArgs {
  const int32_t* input;
  int64_t N;
  int V, d;
  int32_t* count; int32_t* start; int32_t* fill; int32_t* bucket;
  const float* dx; int64_t lddx;
  float* grad; int64_t ldgrad;
};
hipError_t launch_tf_emb_grad(const TfEmbGradArgs& a, hipStream_t s);

}  // namespace erase
