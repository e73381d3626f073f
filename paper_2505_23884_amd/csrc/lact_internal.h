// Internal interface between the host orchestrator (lact_api.hip) and the
// gfx950 kernels (lact_kernels.hip). Not installed; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lact {

constexpr int kMaxDim = 4096;     // envelope for d and h
constexpr int kMaxSplit = 64;     // split-K ways of the gradient contraction

// Operand of one contraction, as seen from a (batch, head) instance.
//   kmajor: element (row r, k) at base + r*ld + k      (row-major [rows x K])
//   mn    : element (row r, k) at base + k*ld + r      (row-major [K x rows])
struct Operand {
  const void* base;     // element (0, 0) of instance 0
  int64_t ld;           // leading dimension, elements
  int64_t inst_stride;  // elements between instances
};

// ---- first launch of a chunk: apply GEMM-1 and/or the key forward ----------
enum FwdKind : int { FWD_APPLY = 0, FWD_UPDATE = 1 };

struct FwdSeg {
  int kind;
  int nblocks;          // instances * tiles_m * tiles_n
  int tiles_m, tiles_n; // hidden tiles (output rows), token tiles
  int64_t rows;         // tokens in this segment
  Operand a0, a1;       // APPLY: q;  UPDATE: k, v            (token-major, kmajor)
  void* out0;           // APPLY: hidden of the queries [rows x h]
  void* out1;           // UPDATE: eta*hidden, eta*dz1, eta*dz3 (token-major)
  void* out2;
  void* out3;
  int64_t out_inst;     // elements between instances of each output
  const float* eta;     // UPDATE: learning rate(s) of token row 0
  int64_t eta_inst;     // floats between instances
  int eta_stride;       // floats per token: 1 (one rate) or 3 (lr1, lr2, lr3 for W1, W2, W3)
  // UPDATE, or nullptr: Z1 = K W1^T, Z3 = K W3^T and D = V W2 themselves
  // (token-major [tokens x h], io dtype, keep_inst elements between
  // instances), kept for the backward's reverse of the same update
  void* keep[3];
  int64_t keep_inst;
};

struct FwdArgs {
  FwdSeg seg[2];
  int nseg;
  int total_blocks;
  int d, h;
  Operand w1, w3;       // h x d, kmajor (operand copies of the fast weight)
  Operand w2;           // d x h; the key forward reads it as an mn operand
  bool narrow;          // 128 x 128 tiles, two workgroups per CU (16-bit, d <= 128)
};

// ---- second launch: apply GEMM-2 and/or the gradient contractions ---------
enum BwdKind : int { BWD_OUT = 0, BWD_GRAD13 = 1, BWD_GRAD2 = 2, BWD_GRAD_UPD = 3 };

struct BwdSeg {
  int kind;
  int nblocks;
  int tiles_m, tiles_n;
  int nsplit;           // GRAD: split-K ways over tokens
  int64_t rows;         // OUT: tokens; GRAD: tokens of the chunk
  int64_t split_len;    // GRAD: tokens per split (multiple of 32)
  Operand a0, a1, b0;   // see lact_kernels.hip for each kind
  void* out;            // OUT: o rows; GRAD: fp32 partials
  int64_t out_inst;     // elements between instances
  int64_t out_split;    // GRAD: elements between splits
  int64_t out_off;      // GRAD2: offset of its matrix in an instance's partials
  const float* row_scale;  // OUT (or nullptr): token t's row is scaled by row_scale[inst * scale_inst + t]
  int64_t scale_inst;
  int64_t klen;         // OUT: contraction length (0: the launch's h)
  // GRAD_UPD (16-bit I/O, whole rows per tile, no split): the gradients of
  // W1 (a0 = eta dz1, b0 = K), W3 (a1 = eta dz3, b0) and W2 (a2 = V,
  // b1 = eta hidden) and the weight update in one pass; tiles_m counts the
  // row tiles of W1, W3 and W2 of one instance, in that order.
  Operand a2, b1;
  float* W[3];          // GRAD_UPD: fp32 state (W1, W2, W3), updated in place
  void* Wb[3];          // GRAD_UPD: bf16 operand copies of the updated state
  float* M[3];          // GRAD_UPD with momentum (else nullptr): the state, updated in place
  const float* bbar;    // chunk-mean momentum factor of instance i at bbar[i * bbar_stride]
  int bbar_stride;
  // GRAD13 / GRAD2 without split (else nullptr): each tile's sum of squares of
  // its gradient block, at sumsq[(inst * spi + j) * sumsq_stride + tile] for
  // matrix j (GRAD13: W1 and W3, j = 0 and 2; GRAD2: j = sumsq_j)
  float* sumsq;
  int sumsq_stride, sumsq_j, spi;
};

// Segments per k_bwd launch: independent products of one chunk's reverse
// share a launch, so that the CUs one product's tiles leave idle take the
// others' (up to two gradient pairs and three output products).
constexpr int kMaxBwdSeg = 7;
struct BwdArgs {
  BwdSeg seg[kMaxBwdSeg];
  int nseg;
  int total_blocks;
  int d, h;
  int narrow;           // 16-bit I/O with d <= 128: the narrow tile shapes (bwd_tile)
};

// ---- weight update ----------------------------------------------------------
struct UpdArgs {
  float* W[3];          // fp32 state W1 [h x d], W2 [d x h], W3 [h x d]
  const float* Wsrc[3]; // where the state before the update is read (nullptr: W itself, in place)
  void* Wb[3];          // operand copies (bf16 mode) or nullptr
  const float* step;    // summed (or split) step, layout [split][inst][3][d*h]
  int nsplit;
  int64_t step_split;   // elements between splits
  int BH, d, h;
  int nmat;             // fast-weight matrices per instance: 3 (SwiGLU) or 1 (linear, d x d with h = d)
  int rows_total;       // BH * (2h + d), or BH * d
  // momentum (nullptr M: none): M_j <- bbar * M_j + g_j, and the update uses M
  float* M[3];          // fp32 momentum, same layout as W
  const float* bbar;    // chunk-mean momentum factor of instance i at bbar[i * bbar_stride]
  int bbar_stride;
};

// ---- Muon: Newton-Schulz on the three gradients of every instance ----------
// Matrices live in "slots" s = inst*3 + j (j = 0: W1, 1: W2, 2: W3), each in
// its stored orientation Y [r x c] (W1, W3: h x d; W2: d x h). The iteration
// runs on the wide orientation of Y:
//   wide (r <= c):  A = Y Y^T,  B = A (c A + b I),  Y <- a Y + B Y
//   tall (r >  c):  A = Y^T Y,  B = A (c A + b I),  Y <- a Y + Y B
// Each product is computed in "tile space", the transpose of what is stored
// (NsSeg M, N are tile-space rows and columns): A and B are symmetric; for
// the update, tile rows are the columns of Y and tile columns its rows.
enum NsKind : int { NS_GRAM_K = 0, NS_GRAM_MN = 1, NS_POLY = 2, NS_UPD_BY = 3, NS_UPD_YB = 4 };

struct NsSeg {
  int kind;
  int nblocks;
  int tiles_m, tiles_n;
  int group;            // matrices per instance in this segment (1 or 2)
  int slot_off[2];      // j of each matrix of the group
  int M, N, K;          // output rows, output columns, contraction length
  int ldy;              // columns c of the stored Y
  int tri;              // symmetric product (16-bit operands, 128 x 128 tiles
                        // only): tiles of the upper triangle, the off-diagonal
                        // ones also writing their mirror
};

struct NsArgs {
  NsSeg seg[2];
  int nseg;
  int total_blocks;
  float* Y32;           // fp32 iterate (in place), slot stride ystride
  int spi;              // slots (matrices) per instance: 3 or 1
  const void* Yin;      // operand copy read this iteration (fp16 or fp32)
  void* Yout;           // operand copy written this iteration (nullptr after the last)
  void* Ab;             // Gram operand copy, slot stride astride
  void* A2b;            // c A + b I (the polynomial's second factor), same layout
  void* Bb;             // polynomial operand copy
  int64_t ystride, astride;
  int m;                // Gram size min(d, h)
  float ca, cb, cc;     // quintic coefficients
};

// Last Newton-Schulz step fused with the weight update (square matrices of
// side m <= 512, 16-bit operands): X5 = a X4 + B X4 for 128 whole rows per
// workgroup, then U = W + X5, W <- U ||W_row|| / ||U_row|| and the bf16 copy.
struct NsFinalArgs {
  const void* Bb;       // polynomial B per slot (fp16, m x m), slot stride astride
  const void* Yin;      // X4 per slot (fp16, m x m), slot stride ystride
  const float* Y32;     // X4 per slot (fp32)
  float* W[3];          // fp32 state of matrix j (instance stride ystride)
  void* Wb[3];          // bf16 operand copies of matrix j
  int spi;              // slots per instance (3, or 1 for the linear fast weight)
  int m;                // side of every matrix
  int64_t ystride, astride;
  int nblocks;          // slots * row tiles
  float ca;             // the quintic's a
};

struct NsPrepArgs {
  const float* part;    // gradient partials [split][inst][3][d*h]
  int nsplit;
  int64_t part_split;   // elements between splits
  float* Y32;           // summed gradient, [inst*spi + j][d*h]
  int spi;              // slots per instance
  float* sumsq;         // per-slot, per-block partial sums of squares
  int nslots;
  int64_t dh;
  int blocks_per_slot;  // blocks of 4096 elements per slot
  // momentum (nullptr M: none); M and the iterate take M <- bbar * M + g first
  float* M[3];
  const float* bbar;
  int bbar_stride;
  // Without split and momentum the gradient tiles leave their sums of squares
  // in sumsq (sum_n[j] entries per slot of matrix j) and k_ns_scale reads the
  // gradient itself from src; nullptr src: Y32 and blocks_per_slot entries
  // (filled by k_ns_prep)
  const float* src;
  int sum_n[3];
};

// Chunk means of the per-token momentum factor: for chunks c in [0, nchunks),
// bbar[i * stride + c] = mean of beta[i * n_kv + t] over t in
// [t0 + c * chunk, min(t0 + (c + 1) * chunk, end)).
constexpr int kBetaBatch = 32;   // chunks per launch (bbar holds BH * kBetaBatch)
struct BetaArgs {
  const float* beta;    // [BH][n_kv]
  int64_t n_kv, chunk;
  int64_t t0, end;      // first token of chunk 0; bound of the last chunk
  int nchunks;          // the forward's batches: <= kBetaBatch; the backward: every chunk
  int BH;
  float* bbar;
  int stride;
};

// Whole Newton-Schulz iteration of small matrices, one workgroup per matrix:
// Gram size m <= 128 and long side n <= 256 (fp16 operands).
constexpr int kNsFusedM = 128, kNsFusedN = 256;
// Quintic Newton-Schulz coefficients (a, b, c) of Muon (App. A, Details of Muon):
// X <- a X + b (X X^T) X + c (X X^T)^2 X
constexpr float kNsA = 3.4445f, kNsB = -4.7750f, kNsC = 2.0315f;
// Muon divides the gradient by ||G||_F + kNsEps, so a zero gradient gives a zero step.
constexpr float kNsEps = 1e-7f;
struct NsFusedArgs {
  // X0 = G / (||G||_F + eps), G the sum of nsplit fp32 partials part_split
  // elements apart (slot stride ystride); steps quintic iterations; then the
  // weight update U = W + X, W <- U ||W_row|| / ||U_row|| with the bf16 copy
  // (W, Wb: the fast weights, instance stride ystride)
  const float* src;
  int nsplit;
  int64_t part_split;
  float eps;
  int spi;              // slots per instance
  int64_t ystride;
  int group;            // matrices per instance in this launch (1 or 2)
  int slot_off[2];      // j of each matrix of the group
  int rows, cols;       // stored orientation Y [rows x cols]
  int nblocks;          // instances * group
  int steps;
  float ca, cb, cc;     // quintic coefficients
  float* W[3];
  void* Wb[3];
};

// ---- the layer's prologue and output norm (lact_io.hip) ---------------------
struct PrologueArgs {
  const void* qkv;      // [B, L, 3, H, hd] io dtype
  const float* lr_raw;  // [B, L, H, R]
  const float* beta_raw;   // [B, L, H] or nullptr
  float lr_bias;
  void *q, *k, *v;      // [B*H, L, hd], [B*H, n_kv, hd] x 2
  float* eta;           // [B*H, n_kv, R]
  float* beta;          // [B*H, n_kv] or nullptr
  int B, H, hd, R;
  int64_t L, n_kv;
  int group;            // set by the launcher
};
struct RmsArgs {
  const void* o;        // [B*H, L, hd]
  const float* weight;  // [H, hd] or nullptr
  void* y;              // [B, L, H, hd]
  float eps;
  int B, H, hd;
  int64_t L;
  int group;            // set by the launcher
};
hipError_t launch_prologue(PrologueArgs a, bool io_bf16, hipStream_t s);
hipError_t launch_rmsnorm_out(RmsArgs a, bool io_bf16, hipStream_t s);
// Reverse of the prologue: from the cotangents of q, k, v, eta (and beta),
// those of the projections, the raw rates (and the raw momentum logits).
struct PrologueBwdArgs {
  const void* qkv;         // [B, L, 3, H, hd] io dtype
  const float* lr_raw;     // [B, L, H, R]
  const float* beta_raw;   // [B, L, H] or nullptr
  float lr_bias;
  const void *dq, *dk, *dv;   // [B*H, L, hd], [B*H, n_kv, hd] x 2
  const float* deta;       // [B*H, n_kv, R]
  const float* dbeta;      // [B*H, n_kv] or nullptr (with beta_raw and dbeta_raw)
  void* dqkv;              // [B, L, 3, H, hd]
  float* dlr_raw;          // [B, L, H, R]
  float* dbeta_raw;        // [B, L, H] or nullptr
  int B, H, hd, R;
  int64_t L, n_kv;
  int group;               // set by the launcher
};
hipError_t launch_prologue_bwd(PrologueBwdArgs a, bool io_bf16, hipStream_t s);
// Reverse of the output RMSNorm: do from dy, and with dweight its cotangent
// through a second pass (r: B*L*H floats of per-vector scales, part: the
// pass's partial sums, rms_dw_splits(...) * H * hd floats).
struct RmsBwdArgs {
  const void* o;           // [B*H, L, hd]
  const float* weight;     // [H, hd] or nullptr
  const void* dy;          // [B, L, H, hd]
  void* d_o;               // [B*H, L, hd]
  float* dweight;          // [H, hd] or nullptr
  float* r;                // scratch [B*L*H] (with dweight)
  float* part;             // scratch (with dweight)
  float eps;
  int B, H, hd;
  int64_t L;
  int group;               // set by the launcher
};
int rms_dw_splits(int B, int64_t L, int H, int hd);
hipError_t launch_rmsnorm_out_bwd(RmsBwdArgs a, bool io_bf16, hipStream_t s);

// Workgroup tile of a contraction kind: output rows x output columns, threads.
struct TileShape {
  int rows, cols, threads;
};
TileShape fwd_tile(int kind, bool io_bf16, bool narrow);   // rows = hidden units, cols = tokens
TileShape bwd_tile(int kind, bool io_bf16, bool narrow);   // OUT: features x tokens; GRAD13:
                                                           // hidden x features; GRAD2: features x hidden
TileShape ns_tile(bool fp16, bool big);       // tile-space rows x columns of the NS products
TileShape grad_upd_tile();                    // GRAD_UPD: rows of W x all columns (bf16)

// Launchers (io_bf16 selects bf16 MFMA operands, otherwise fp32).
hipError_t launch_fwd(const FwdArgs& a, bool io_bf16, hipStream_t s);
hipError_t launch_bwd(const BwdArgs& a, bool io_bf16, hipStream_t s);
hipError_t launch_update(const UpdArgs& a, bool io_bf16, hipStream_t s);
// out[i][t] = eta[i][t] * k[i][t] for t < n (rows of d elements, io dtype).
hipError_t launch_scale_rows(const void* k, const float* eta, void* out, int BH, int64_t n, int d, int64_t k_inst,
                             int64_t eta_inst, int64_t out_inst, bool io_bf16, hipStream_t s);
// W[1] == nullptr: one matrix (W[0] -> Wb[0]).
hipError_t launch_prep(const float* const W[3], void* const Wb[3], int BH, int d, int h,
                       hipStream_t s);
// Newton-Schulz operand copies are fp16 (bf16 I/O: 4x finer rounding than bf16
// at the same MFMA rate; the iterates are O(1)) or fp32 (fp32 I/O).
hipError_t launch_ns(const NsArgs& a, bool fp16, bool big, hipStream_t s);
hipError_t launch_ns_final(const NsFinalArgs& a, hipStream_t s);
TileShape ns_final_tile();   // k_ns_final: rows per workgroup x the largest side
hipError_t launch_ns_prep(const NsPrepArgs& a, hipStream_t s);
hipError_t launch_ns_scale(const NsPrepArgs& a, void* Yb, bool fp16, float eps, hipStream_t s);
hipError_t launch_ns_fused(const NsFusedArgs& a, hipStream_t s);
hipError_t launch_ns_fused_pair(const NsFusedArgs& a0, const NsFusedArgs& a1, hipStream_t s);
// The same with the output tiles of one chunk (out: one BWD_OUT segment, narrow
// shapes) in the launch; the Newton-Schulz writes the copies of the other set.
hipError_t launch_ns_fused_pair_out(const NsFusedArgs& a0, const NsFusedArgs& a1, const BwdArgs& out,
                                    hipStream_t s);
hipError_t launch_beta_mean(const BetaArgs& a, hipStream_t s);
// Zero rows [r0, r1) of every instance of an output of `rows` rows of row_bytes
// (a multiple of 16) each.
// ---- backward: the steps between the OUT / GRAD contractions --------------
// A set of fp32 split partials of a [R x L] matrix: element (inst, r, c) of
// split s at p[s * split + inst * inst + r * L + c], summed over s < n
// (p == nullptr or n == 0: no set).
struct PartSet {
  const float* p;
  int n;
  int64_t split, inst;
  float sign;   // factor of the sum (0: 1)
};

// Reverse of W' = (n / u) U, U = W + sum P, per row of a [R x L] matrix.
struct VjpArgs {
  const float* W; int64_t w_inst;     // weights entering the chunk
  PartSet P;                          // U = W + sum P (the negated chunk gradient)
  PartSet pre[2];                     // added to the cotangent before the reverse
  PartSet post;                       // added after it
  float* G; int64_t g_inst;           // cotangent of W' in, of W out (in place)
  void* Ub; int64_t ub_ld, ub_inst;   // cotangent of U in the operand type, row-major (or nullptr)
  void* UT; int64_t ut_ld, ut_inst;   // the same, transposed (or nullptr)
  float* U32; int64_t u32_inst;       // the same in fp32, row-major with rows of L (or nullptr)
  int BH, R, L;
};

// Up to three matrices' reverses in one launch (rows of the longest up to 4096).
hipError_t launch_vjp(const VjpArgs* a, int n, bool io_bf16, hipStream_t s);
// Operand copies of fp32 [R x L] matrices (w_inst apart) in the operand
// type: dst = W (dst[r * ld + c], dst_inst apart) and/or dstT = W^T
// (dstT[c * ldT + r], dstT_inst apart), either one may be nullptr; up to
// kMaxCopies matrices in one launch.
struct CopySeg {
  const float* W; int64_t w_inst;
  int R, L;
  void* dst; int64_t ld, dst_inst;
  void* dstT; int64_t ldT, dstT_inst;
  int nsum;                 // source splits summed (0 or 1: one)
  int64_t split;            // floats between source splits
  float sign;               // factor of the sum (0: 1)
};
constexpr int kMaxCopies = 8;
hipError_t launch_copies(const CopySeg* c, int n, int BH, bool io_bf16, hipStream_t s);
// The same with fp32 copies.
hipError_t launch_copies_f32(const CopySeg* c, int n, int BH, hipStream_t s);

// ---- reverse of Newton-Schulz (slots of wide [m x n] fp32 matrices) --------
// The k_bwd kinds with fp16 operands (fp16 OUT results, fp32 GRAD partials).
// a.narrow: the narrow kinds (128-row GRAD2 tiles)
hipError_t launch_bwd_f16(const BwdArgs& a, hipStream_t s);
// out[s] = sum over len elements of x[s] * y[s] (slot s), in a fixed order
// (32 workgroups per slot, then their partials in order).
hipError_t launch_slot_dot(const float* x, const float* y, int S, int64_t len, float* out, float* part,
                           hipStream_t s);   // part: S * 32 floats of scratch
// Elementwise over S slots of len floats (x, y, p1, p2 fp32; sc, sc2 per slot):
//   mode 0: out = x / (sqrt(sc) + eps)
//   mode 1: out = a x + p1 (+ p2 when given)
//   mode 2: out = x / (sqrt(sc) + eps) - sc2 / ((sqrt(sc) + eps)^2 sqrt(sc)) y
// into out32 and/or its fp16 copy out16.
struct NsLinArgs {
  int mode;
  const float* x; const float* y; const float* p1; const float* p2;
  const float* sc; const float* sc2;
  float a, eps;
  float* out32; _Float16* out16;
  float* outc32;   // an fp32 operand copy (fp32 I/O) in place of out16
  int S; int64_t len;
};
hipError_t launch_ns_lin(const NsLinArgs& a, hipStream_t s);
// out = alpha X + beta (Y + Y^T) per slot of fp16 [m x m] matrices (X may be nullptr).
hipError_t launch_sym(const _Float16* X, float alpha, const _Float16* Y, float beta, _Float16* out, int S, int m,
                      hipStream_t s);
// The same for fp32 slots (fp32 I/O).
hipError_t launch_sym32(const float* X, float alpha, const float* Y, float beta, float* out, int S, int m,
                        hipStream_t s);
// G = base + sum of the sets over BH instances of RL floats each (RL a
// multiple of 4); base: 0 (mode 0), init (mode 1) or G itself (mode 2).
hipError_t launch_accum(float* G, int64_t g_inst, const float* init, int64_t i_inst, int mode, PartSet s0, PartSet s1,
                        int BH, int64_t RL, hipStream_t s);
// Momentum reverse of one chunk (M' = bbar M + g): U holds minus the
// cotangent that reaches M' through the update's step ([inst][nmat][dh]); R
// (per matrix [BH][dh]) the cotangent carried from later chunks. With
// dM' = R - U: U <- -dM' (the gradient's cotangent, negated), R <- bbar dM',
// and part[inst * nblk + b] the block's share of <dM', M> (M per matrix).
struct MomBwdArgs {
  float* U;
  float* R[3];
  const float* M[3];
  const float* bbar; int64_t bbar_inst;
  float* part;
  int BH, nmat, nblk;
  int64_t dh;
};
hipError_t launch_mom_bwd(const MomBwdArgs& a, hipStream_t s);
// dbeta[inst * n_kv + t] = (sum of the instance's nblk partials) / n for t < n.
hipError_t launch_mom_dbeta(const float* part, int nblk, int BH, float* dbeta, int64_t n_kv, int64_t n, hipStream_t s);
// M'[inst] = bbar[inst * bbar_inst] M[inst] - (sum of the nsplit partials P), dh floats per instance.
hipError_t launch_mom_adv(const float* M, const float* bbar, int64_t bbar_inst, PartSet P, float* Mout, int BH,
                          int64_t dh, hipStream_t s);
// Linear fast weight, per key token of a chunk: dv = eta Y (Y in dv on
// entry), deta = v . Y.
hipError_t launch_lin_tokens(const void* V, const float* eta, void* dv, float* deta, int BH, int64_t n, int d,
                             int64_t tok_inst, int64_t eta_inst, bool io_bf16, hipStream_t s);

// SwiGLU fast weight, per key token of a chunk (rows of h): from Z1 = K W1^T,
// Z3 = K W3^T, C = V W2, X1 = K U1^T, X3 = K U3^T, Y2 = V U2 (U: the update's
// cotangent) and eta, the operands Pk = [R3 | R1 | dZ1 | dZ3] and
// Pv = [eta A | dC] of the next contractions and deta.
struct SwigluRowsArgs {
  const void* Z1; const void* Z3; const void* C; const void* X1; const void* X3; const void* Y2;
  int64_t in_inst;                    // elements between instances of the six [n x h] inputs
  int64_t z_inst;                     // the same for Z1, Z3 and C when nonzero (else in_inst)
  const float* eta; int64_t eta_inst;  // tokens between instances; eta_cols rates per token (1, or 3 per matrix)
  int eta_cols;                       // deta has the same layout
  void* Pk; int64_t pk_inst;          // [n x 4h]
  void* Pv; int64_t pv_inst;          // [n x 2h]
  float* deta;
  int BH; int64_t n; int h;
};
hipError_t launch_swiglu_rows(const SwigluRowsArgs& a, bool io_bf16, hipStream_t s);
// SwiGLU apply, per query token: from Zq1 = Q W1^T, Zq3 = Q W3^T, Dh = dO W2,
// Pq = [dZq1 | dZq3] ([n x 2h]) and Hq = SiLU(Zq1) o Zq3 ([n x h]).
hipError_t launch_swiglu_apply_rows(const void* Z1, const void* Z3, const void* Dh, int64_t in_inst, void* Pq,
                                    int64_t pq_inst, void* Hq, int64_t hq_inst, int BH, int64_t n, int h, bool io_bf16,
                                    hipStream_t s);
hipError_t launch_zero_rows(void* out, int BH, int64_t row_bytes, int64_t rows, int64_t r0, int64_t r1,
                            hipStream_t s);
// x[i * inst + off + j] = 0 for j in [0, count), instances i in [0, BH).
hipError_t launch_zero_f32(float* x, int BH, int64_t inst, int64_t off, int64_t count, hipStream_t s);
constexpr int kNsBlockElems = 4096;

}  // namespace lact
