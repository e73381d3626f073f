// Internal interface between the host orchestrator (lact_api.hip) and the
// gfx950 kernels (lact_kernels.hip). Not installed; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lact {

constexpr int kTile = 128;        // output tile edge of every MFMA contraction
constexpr int kThreads = 256;     // 4 waves of 64 lanes
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
  int tiles_m, tiles_n; // token tiles, hidden tiles
  int64_t rows;         // tokens in this segment
  Operand a0, a1;       // APPLY: q;  UPDATE: k, v            (token-major, kmajor)
  void* out0;           // APPLY: hidden of the queries [rows x h]
  void* out1;           // UPDATE: eta*hidden, eta*dz1, eta*dz3 (token-major)
  void* out2;
  void* out3;
  int64_t out_inst;     // elements between instances of each output
  const float* eta;     // UPDATE: per-token learning rate of token row 0
  int64_t eta_inst;
};

struct FwdArgs {
  FwdSeg seg[2];
  int nseg;
  int total_blocks;
  int d, h;
  Operand w1, w3;       // h x d, kmajor (operand copies of the fast weight)
  Operand w2;           // d x h; the key forward reads it as an mn operand
};

// ---- second launch: apply GEMM-2 and/or the gradient contractions ---------
enum BwdKind : int { BWD_OUT = 0, BWD_GRAD13 = 1, BWD_GRAD2 = 2 };

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
};

struct BwdArgs {
  BwdSeg seg[3];
  int nseg;
  int total_blocks;
  int d, h;
};

// ---- weight update ----------------------------------------------------------
struct UpdArgs {
  float* W[3];          // fp32 state W1 [h x d], W2 [d x h], W3 [h x d]
  void* Wb[3];          // operand copies (bf16 mode) or nullptr
  const float* step;    // summed (or split) step, layout [split][inst][3][d*h]
  int nsplit;
  int64_t step_split;   // elements between splits
  int BH, d, h;
  int rows_total;       // BH * (2h + d)
};

// Launchers (io_bf16 selects bf16 MFMA operands, otherwise fp32).
hipError_t launch_fwd(const FwdArgs& a, bool io_bf16, hipStream_t s);
hipError_t launch_bwd(const BwdArgs& a, bool io_bf16, hipStream_t s);
hipError_t launch_update(const UpdArgs& a, bool io_bf16, hipStream_t s);
hipError_t launch_prep(const float* const W[3], void* const Wb[3], int BH, int d, int h,
                       hipStream_t s);

}  // namespace lact
