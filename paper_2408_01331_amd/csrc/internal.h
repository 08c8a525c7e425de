// Device-side problem descriptors shared by the host planner (un_api.cpp) and
// the gfx950 kernels (kernels.hip). Everything here is plain data: the planner
// fills these tables once in un_create and uploads them into the arena; a step
// only launches kernels over them.
#pragma once
#include <stdint.h>

#include <hip/hip_runtime.h>

namespace un {

// Storage element types: fp32 or bf16 (raw 16-bit pattern, round-to-nearest-even).
typedef uint16_t bf16_t;

// ---------------------------------------------------------------------------
// Grouped GEMM:  C[m][n] = sum_k A[m][k] * B[n][k]
// Each operand is row-major (element (r, k) at base[r*ld + k], k contiguous)
// or k-major (element (r, k) at base[k*ld + r]). A k-major operand is staged
// in LDS as it lies in memory and turned into MFMA operands by the LDS
// transpose reads of gfx950, so no layer keeps a transposed copy of its
// weights, activations or gradients:
//   forward  Y[b][o]  = sum_i X[b][i] W[o][i]    A = X row-major,  B = W row-major
//   dgrad    dX[b][i] = sum_o G[b][o] W[o][i]    A = G row-major,  B = W k-major
//   wgrad    dW[o][i] = sum_b G[b][o] X[b][i]    A = G k-major,    B = X k-major
// The wgrad's B loader reads 1 in column n == nsplit (for every k < K): that
// column of the product is the bias gradient sum_b G[b][o].
// ---------------------------------------------------------------------------
enum OpLayout : int32_t { OP_ROW = 0, OP_KMAJ = 1 };

enum Epi : int32_t {
  EPI_FWD = 0,     // + bias, optional ReLU, store C (T)
  EPI_LOGITS = 1,  // + bias, store C as fp32
  EPI_DGRAD = 2,   // optional ReLU' mask from `mask` (row-major [m][n], keep where > 0), store C (T)
  EPI_WGRAD = 3,   // store C as fp32 for n < nsplit; column nsplit -> dbias[m]
  EPI_WPART = 4    // split-K weight gradient: the fp32 partial sums of k-chunk `split`
                   // (bias column included) to ws[split][m][n]; a reduction adds the
                   // splits in order and applies the update
};

struct GemmProb {
  const void* A;
  const void* B;
  int64_t lda, ldb;
  int32_t M, N, K;
  int32_t epi, relu;
  int32_t amode, bmode;       // OpLayout of A and B
  int32_t tiles_n;
  int32_t nsplit;
  int32_t model;              // WGRAD: the model whose learning rate applies (single-model problems)
  void* C;                    // WGRAD: gradient dW [m][ldc] (stored only when gradients are kept)
  int64_t ldc;
  const float* bias;
  const void* mask;
  int64_t ldmask;
  float* dbias;               // WGRAD: bias gradient (kept gradients only)
  // WGRAD with the SGD update fused into the epilogue:
  //   W[m][n] <- fma(-lr, dW[m][n], W[m][n]) (fp32 master, row stride ldc),
  //   Wb[m][n] <- bf16(W) (bf16 mode), bmaster[m] <- fma(-lr, db[m], bmaster[m]).
  float* W;
  void* Wb;
  float* bmaster;
  const int32_t* row_model;   // WGRAD of the concatenated first layers: model of each row m (else null)
  // LOGITS with softmax-CE fused (N <= the tile width, so a tile holds whole
  // rows): C/ldc is the gradient dL/dz (storage type) of model `model`, and
  // the tile's summed row losses go to ce_part[m-tile]. Null: C is the fp32
  // logits and a separate CE pass follows.
  float* ce_part;
  // labels of the fused softmax-CE: labels + lab_shared (the model's input
  // group row) or labels + lab_own (its own row, per-model labels)
  int32_t lab_shared, lab_own;
  // Skip connection (residual blocks), row-major [m][n] in the storage type,
  // added in fp32 before the ReLU (FWD) or before the ReLU' mask (DGRAD):
  // FWD: the block's input x; DGRAD: the gradient at the block's output. Null: none.
  const void* R;
  int64_t ldr;
  // optimizer state (same layouts as W and bmaster; null for plain SGD):
  // momentum buffer or Adam's first moment, and Adam's second moment
  float* s1;
  float* s2;
  float* sb1;
  float* sb2;
  // WPART: k-blocks [split * kchunk, (split + 1) * kchunk) of `splits` per
  // tile (tile map entry: split * tiles + tile); partials at ws (a workspace
  // buffer: the step's byte offset added), row stride ldws floats
  int32_t splits, kchunk;
  float* ws;
  int64_t ldws;
};

// ---------------------------------------------------------------------------
// Implicit-GEMM convolution (NHWC activations, stride 1, square kernel).
// Pooled outputs are indexed by window w = (n*PH + ph)*PW + pw and the conv
// output pixels feeding a pool are ordered m = 4*w + (dy*2 + dx), so the four
// members of one 2x2 window are four consecutive GEMM rows.
//   fwd:   C[m][o]  = sum_{(u,v,c)} Xpatch[m][(u,v,c)] * W[o][(u,v,c)]
//   dgrad: C[m][c]  = sum_{(u,v,o)} dZ[n, y-u+pad, x-v+pad, o] * WT[c][(u,v,o)]
//          (m = (n*H + y)*W + x over the conv's input pixels)
//   wgrad: C[o][j]  = sum_{pixels} dZ[pix][o] * Xpatch[pix][j], j = (u,v,c);
//          column j == KH*KW*C is the bias gradient. Split over pixel ranges;
//          partial sums go to ws[split][o][j] and are reduced in split order.
// dZ is never stored: it is gathered from the pooled gradient G[w][o] (which
// already carries this block's ReLU' mask) and the window argmax.
//
// Halo tiling (fwd and dgrad, when the row-tile geometry fits, halo != 0): a
// tile of BM rows is `imgs` whole images or `tr` whole rows of one image of
// the pass's pixel space (fwd: conv output OHxOW; dgrad: conv input HxW). The
// workgroup stages the operand rows that tile reads - `hr` rows x `hc`
// columns per image, channels in blocks of `cb` (LDS stride `cs`) - once per
// channel block in LDS, and reads every kernel tap from there; k runs over
// (channel block, tap, channel in block). Weight columns keep the (tap, c)
// order, so a k-block gathers its weight columns by tap.
// ---------------------------------------------------------------------------
struct ConvProb {
  int32_t Nb, C, H, W, O, KH, pad, OH, OW, PH, PW;
  int32_t pool, relu, prev_relu;
  int32_t M, N, K;            // GEMM sizes of this pass
  int32_t tiles_m, tiles_n, splits, kchunk;
  int32_t halo, tr, imgs, hr, hc, cb, cs;  // halo tiling (see above)
  int32_t bm, bn;                          // halo tile shape
  // forward halo passes with one channel block: consecutive m-tiles of one
  // n-column per workgroup (weights and tap tables loaded once, the next
  // tile's rows fetched during this tile's epilogue); else 1
  int32_t mt;
  // fl(1/d) (correctly rounded) for the halo tile's small divisors, computed
  // once on the host: tile rows per image and per image row (pooled forward:
  // windows), KH, 16-byte chunks per position of a full and of the last
  // channel block, staged positions per image (hr * hc) and hc
  float rc_img, rc_row, rc_kh, rc_cpt, rc_cpt_last, rc_plane, rc_hc;
  const void* X;              // conv input, NHWC, channel stride C
  const void* Wt;             // fwd: W [O][ldw]; dgrad: WT [C][ldw]
  int64_t ldw;
  const float* bias;          // fwd
  void* P;                    // fwd output (pooled or not), [pixel][O]
  uint8_t* amax;              // fwd: window argmax as the one-hot byte 1 << (dy*2 + dx), [w][O]
  const void* G;              // dgrad/wgrad: gradient at this block's output, [pixel][O]
  const uint8_t* gam;         // its argmax (pool only)
  void* Gprev;                // dgrad output [n*H*W + y*W + x][C]
  float* ws;                  // wgrad partials [splits][O][ldws]
  int64_t ldws;
  // Skip connection (residual blocks; pool == 0, pixel-ordered rows), added in
  // fp32 before the ReLU (fwd: the block's input x [pixel][O]) or before the
  // previous block's ReLU' (dgrad: the gradient at the block's output
  // [pixel][C]). Null: none.
  const void* R;
};

// Split-K reduction of conv weight-gradient partials, in split order, with
// the SGD update fused: W[o][j] <- fma(-lr, dW, W), its bf16 copy and its
// transposed copy WT[c][tap*O + o] (j = tap*C + c) that the conv data gradient
// reads, and the bias from column J.
// dW / db are also stored when gradients are kept (gW / gb non-null).
struct ReduceProb {
  const float* ws;
  int64_t ldws;
  int32_t splits, O, J, C;    // J = KH*KW*C weight columns (+1 bias column in ws)
  int32_t blk_base;
  int32_t model;
  float* gW;
  int64_t ldgw;
  float* gb;
  float* W;                   // master [O][ldgw]
  void* Wb;
  void* WT;
  int64_t ldwt;
  float* bmaster;
  float* s1;                  // optimizer state, as in GemmProb
  float* s2;
  float* sb1;
  float* sb2;
};

// ---------------------------------------------------------------------------
// Self-attention core of one model, per sample b (one workgroup each):
//   forward:  S = Q K^T * scale, P = softmax(S) over the keys, A = P V
//   backward: dP = dA V^T, dS = P * (dP - rowsum(P * dP)), dQ = dS K * scale,
//             dK = dS^T Q * scale, dV = P^T dA
// Q | K | V are the three d-column parts of the in-projection's token rows
// (QKV [B*T][ldq], storage type); A and dA are [B*T][lda]; dQKV has QKV's
// layout; P [B][T][T] fp32 is written by the forward and read by the backward.
// Every output element is one fmaf chain in a fixed order.
// ---------------------------------------------------------------------------
struct AttnProb {
  const void* QKV;
  int64_t ldq;
  void* A;
  int64_t lda;
  const void* dA;
  void* dQKV;
  float* P;
  int32_t T, d, B;
  float scale;
};

// LDS of one workgroup: Q, K, V (and dA) in the storage type (es bytes per
// element) as rows of d plus one 16-byte chunk, and one (two) T x (T + 1)
// fp32 score tiles. The parser's bound takes es = 4.
inline size_t attn_lds_bytes(int T, int d, bool bwd, int es) {
  return (size_t)(bwd ? 4 : 3) * T * (d + 16 / es) * es + (size_t)(bwd ? 2 : 1) * T * (T + 1) * 4;
}

// ---------------------------------------------------------------------------
// Optimizer of one model for one step, computed on the host per step (all
// fields fp32 so that the array travels as plain floats):
//   kind 0  SGD:           w <- fma(-lr, g, w)
//   kind 1  SGD momentum:  b <- fma(b1, b, g);  w <- fma(-lr, b, w)   (b1 = momentum)
//   kind 2  Adam:          m <- fma(b1, m, c1*g);  v <- fma(b2, v, c2*g*g);
//                          w <- w - lr * (m / (sqrt(v) * isb2 + eps))
// with, for Adam at its step t: lr = rate / (1 - beta1^t), c1 = 1 - beta1,
// c2 = 1 - beta2, isb2 = 1 / sqrt(1 - beta2^t).
// ---------------------------------------------------------------------------
struct OptHp {
  float kind, lr, b1, b2, c1, c2, isb2, eps;
};
constexpr int OPT_FLOATS = 8;

// ---------------------------------------------------------------------------
// Softmax cross-entropy of one model: logits [B][ldl] fp32 -> per-model mean
// loss, and dz = (softmax - onehot)/B stored as G [B][ldg].
// Row losses are summed per 32-row chunk, then per model, in a fixed order.
// ---------------------------------------------------------------------------
struct CeProb {
  const float* logits;
  int64_t ldl;
  void* G;
  int64_t ldg;
  int32_t C;
  int32_t model;
  int32_t nchunks;            // loss partials of this model (row chunks or GEMM m-tiles)
  int32_t B;                  // the model's batch (its input group's)
  int32_t lab_shared, lab_own;  // its labels: labels + lab_shared (group row) or + lab_own (own row)
  // split-K logits (nparts > 0): the logits are the partials parts[s][b][c]
  // (row stride ldp, nparts slices of B rows) added in split order, plus
  // bias[c]; the row pass writes them to `logits` first. Else null / 0.
  const float* parts;
  int64_t ldp;
  int32_t nparts;
  const float* bias;
};

// ---------------------------------------------------------------------------
// Multi-tensor SGD over 64x64 tiles of every parameter tensor:
//   W <- fma(-lr, G, W)  (fp32 master), then the copies the GEMMs read:
//   Wb  [r][ldw]          bf16 copy in the same layout (bf16 mode), and
//   WT  [c][j*R + r]      a conv block's transposed copy that its data
//                         gradient reads (T), where the tensor is viewed as
//                         [R][J][Cc] (J = kernel taps).
// With use_grad false only the copies are refreshed (after set/init).
// ---------------------------------------------------------------------------
struct SgdTensor {
  float* W;
  const float* G;
  void* Wb;
  void* WT;
  int64_t ldw, ldwt;
  int32_t R, J, Cc;
  int32_t tiles_r, tiles_c;   // per tap
  int32_t tile_base;
};

// Kernel launch wrappers (kernels.hip). `bf16` selects the storage type.
// `tile_map` holds one (problem index, tile index within the problem) pair of
// int32 per workgroup, in launch order; a pair with problem -1 is padding and
// its workgroup does nothing.
// Learning rates: `lr` for every model, or per model lrv[model] when lrv is
// not null (device array). Labels: labels[b] for every model, or
// labels[model * B + b] when per_model_labels is set.
// `opt` (device, one OptHp per model) replaces lr/lrv when not null.
// bwd: the launch holds data- and weight-gradient problems (k-major operands),
// else forward problems (row-major operands only).
// labels / per_model_labels: the label buffer of the fused softmax-CE; a
// model reads its own row (GemmProb::lab_own) when per_model_labels is set,
// else its input group's row (lab_shared).
// wsoff: byte offset added to every workspace pointer of the descriptors
// (split-K partials GemmProb::ce_part, ConvProb::ws, ReduceProb::ws), so that
// one set of tables serves the arena's workspace (0) or another buffer of the
// same layout.
hipError_t launch_gemm(bool bf16, bool bwd, const GemmProb* probs, const int32_t* tile_map, int ntiles, float lr,
                       const float* lrv, const OptHp* opt, bool keep_grads, const int32_t* labels,
                       bool per_model_labels, int64_t wsoff, hipStream_t s);
hipError_t launch_conv_fwd(bool bf16, const ConvProb* probs, const int32_t* tile_map, int ntiles,
                           hipStream_t s);
hipError_t launch_conv_dgrad(bool bf16, const ConvProb* probs, const int32_t* tile_map, int ntiles,
                             hipStream_t s);
// mode: 0 any layer; 1 pooled, 2 unpooled, both with O and C whole 16-byte vectors
hipError_t launch_conv_wgrad(bool bf16, int mode, const ConvProb* probs, const int32_t* tile_map, int ntiles,
                             int64_t wsoff, hipStream_t s);
// Halo-tiled forward (dgrad = false) or data gradient (dgrad = true); every
// problem of the launch has halo != 0 (either tile shape).
hipError_t launch_conv_halo(bool bf16, bool dgrad, const ConvProb* probs, const int32_t* tile_map, int ntiles,
                            size_t lds_bytes, hipStream_t s);
hipError_t launch_reduce(bool bf16, const ReduceProb* probs, const int32_t* blk_prob, int nblocks, float lr,
                         const float* lrv, const OptHp* opt, bool keep_grads, int64_t wsoff, hipStream_t s);
hipError_t launch_set_values(float* dst, const float* vals, int n, hipStream_t s);
// tile_map: one (problem, sample) pair per workgroup.
hipError_t launch_attn(bool bf16, bool bwd, const AttnProb* probs, const int32_t* tile_map, int nblocks,
                       size_t lds_bytes, hipStream_t s);
// probs: the first nrows problems need the row pass (their CE is not fused
// into the logits GEMM); the loss of every one of the nprobs is finished.
// Partials of model m are at partial + m * pstride; maxB is the largest
// batch of the problems (each has its own, CeProb::B).
// Split-K logit partials (CeProb::parts) are read at parts + wsoff bytes.
hipError_t launch_ce(bool bf16, const CeProb* probs, int nprobs, int nrows, const int32_t* labels,
                     bool per_model_labels, int maxB, float* partial, int pstride, float* losses, int64_t wsoff,
                     hipStream_t s);
// The launch covers tiles [blk0, blk0 + ntiles) of the tile table.
hipError_t launch_sgd(bool bf16, const SgdTensor* t, const int32_t* tile_tensor, int blk0, int ntiles, float lr,
                      bool use_grad, hipStream_t s);
// fp32 NCHW batch -> storage type: NHWC X (optional) and NHWC XC with
// Cs >= C channels (optional; the channels from C on are left untouched).
hipError_t launch_load(bool bf16, const float* x, int B, int C, int H, int W, void* X, void* XC, int Cs,
                       hipStream_t s);

// Tile shapes the planner must agree with.
constexpr int GEMM_BM_BF16 = 128, GEMM_BN_BF16 = 128;
constexpr int GEMM_BM_F32 = 64, GEMM_BN_F32 = 64;
constexpr int GEMM_BK_BF16 = 64, GEMM_BK_F32 = 32;
constexpr int CONV_BM_BF16 = 128, CONV_BN_BF16 = 128, CONV_BK_BF16 = 64;
constexpr int CONV_BM_F32 = 64, CONV_BN_F32 = 64, CONV_BK_F32 = 32;
// bf16 conv weight gradients whose blocks all have at most this many output
// channels run 64-row tiles (launch mode bit WG_NARROW_BIT)
constexpr int CONV_WG_NARROW_BM = 64, WG_NARROW_BIT = 4;
constexpr int SGD_TILE = 64;
constexpr int REDUCE_BLOCK = 256;
constexpr int CE_MAX_BATCH = 1 << 20;
constexpr int CE_ROWS = 32;           // sample rows per softmax-CE block
constexpr int CE_LANES = 8;           // lanes per row
// Halo tiles. Two shapes: wide BM x BN = CONV_BM x CONV_BN, and narrow
// (2*CONV_BM) x (CONV_BN/2) for passes with at most CONV_BN/2 output columns.
// LDS per workgroup: the double-buffered weight stage, two chunk tables of
// HALO_QMAX ints, and the staged rows - halo_elems() elements.
constexpr int HALO_QMAX = 256;
// Threads of a halo workgroup (bf16: 8 waves, fp32: 4) and the 16-byte
// chunks per thread that a multi-tile forward workgroup fetches ahead: its
// staged rows must fit HALO_PF * threads chunks.
constexpr int HALO_NT_BF16 = 512, HALO_NT_F32 = 256, HALO_PF = 4;
constexpr int HALO_LDS_BF16 = 80 * 1024, HALO_LDS_F32 = 52 * 1024;  // two (bf16) / three (fp32) per CU
constexpr int halo_elems(int es, int BN, int BK) {
  return ((es == 2 ? HALO_LDS_BF16 : HALO_LDS_F32) - 2 * HALO_QMAX * 4 - 2 * BN * (BK + 16 / es) * es) / es;
}

// LDS bytes of a halo problem: weight stages, chunk tables and staged rows
// during the main loop; the data gradient's staged output tile in the epilogue.
inline size_t halo_lds_bytes(const ConvProb& p, int es, int BK, bool dgrad) {
  const size_t main = (size_t)2 * p.bn * (BK + 16 / es) * es + 2 * HALO_QMAX * 4 + (size_t)p.imgs * p.hr * p.hc * p.cs * es;
  const size_t epi = dgrad ? (size_t)p.bm * (p.bn + 16 / es) * es : 0;
  return main > epi ? main : epi;
}

}  // namespace un
