// gfx950 kernels of the LaCT fast-weight layer forward.
//
// Every contraction of the path is a batched GEMM tile loop with fp32
// accumulation and a fused epilogue per kind:
//
//   FWD_APPLY   Z^T = W1 Q^T, W3 Q^T          -> hidden SiLU(Z1) o Z3        (apply, §3.1 SwiGLU eq.)
//   FWD_UPDATE  Z^T = W1 K^T, W3 K^T, D^T = (V W2)^T
//               -> eta*hidden, eta*dz1, eta*dz3: the key forward and the
//               backward to the hidden units of grad sum_i eta_i (-f_W(k_i)^T v_i)
//               (§3.1 loss and chunk-gradient eqs.; Alg. 1, update)
//   BWD_OUT     O^T = W2 hidden^T                                  (apply, second matmul)
//   BWD_GRAD13  P1 = (eta dz1)^T K,  P3 = (eta dz3)^T K             (gradient matmuls, -g1, -g3)
//   BWD_GRAD2   P2 = V^T (eta hidden)                              (-g2; the linear
//               fast weight's gradient V^T (eta K), §5.4, with OUT as its apply)
//   BWD_GRAD_UPD  P1, P3, P2 of whole rows (256 < d, h <= 512) followed in the
//               same workgroup by the weight update of those rows, with or
//               without momentum (no Muon, no split): the gradient never goes
//               to memory
// (for d <= 128 both launches have narrow shapes: OUT, GRAD13 and GRAD2 whose
// feature dimension fills the tile, and k_fwd_narrow, whose 128 x 128 tiles
// let two workgroups share a CU)
//   NS_*        Newton-Schulz products (Muon, §3.2; App. A); k_ns_fused and
//               k_ns_fused_pair run the whole iteration of a small matrix in
//               one workgroup
// plus the separate weight update with its row normalisation and momentum
// (k_update, wherever neither the gradient and update kind, k_ns_final nor
// the fused small-matrix Newton-Schulz applies it),
// the Newton-Schulz prologue (k_ns_prep, k_ns_scale), the momentum chunk
// means (k_beta_mean), operand copies (k_prep), eta k (k_scale_rows) and the
// zeroing of uncovered output rows (k_zero_rows).
//
// 16-bit operands (bf16 I/O; fp16 for Newton-Schulz) run on
// v_mfma_f32_32x32x16_{bf16,f16}. A workgroup of WM x WN waves owns a tile of
// (32*MI*WM) x (32*NI*WN) outputs, every wave (32*MI) x (32*NI). Operand tiles
// go from HBM to LDS by raw-buffer DMA (buffer_load_dwordx4 ... lds) into a
// ring of NSTAGE stages of BK K each. An operand is either K-contiguous in HBM
// ("k": row-major [rows x K], kept as BK*2-byte rows in LDS, BK = 64 so that
// every DMA fetches whole 128-byte lines, except in k_fwd_narrow) or row-contiguous ("mn": row-major
// [K x rows], the token-major layout; BK = 32 K rows in LDS, read with
// ds_read_b64_tr_b16, which returns MFMA fragments of the transposed operand).
// fp32 I/O runs on v_mfma_f32_32x32x2_f32 with a register-staged double
// buffer (the transposition of mn operands happens in registers there).
#include "lact_internal.h"

namespace lact {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

constexpr int kRowBytes = 64;
constexpr int kTileBytes = 128 * kRowBytes;   // a 128-row operand tile (fp32 path)

template <typename T> struct Tr;
template <> struct Tr<__bf16> {   // 32 K per tile, 8 elements per 16 bytes
  static constexpr int BK = 32, E = 8, KG = 8;
};
template <> struct Tr<_Float16> { // fp16 operands (Newton-Schulz): as bf16
  static constexpr int BK = 32, E = 8, KG = 8;
};
template <> struct Tr<float> {    // 16 K per tile, 4 elements per 16 bytes
  static constexpr int BK = 16, E = 4, KG = 4;
};

// LDS byte offset of 16-byte chunk `chunk` (0..3) of row `row` of a
// K-contiguous tile. The XOR with row bits 2-3 keeps the 16-lane groups that
// serve one MFMA fragment read (16 consecutive rows, one chunk) free of bank
// conflicts (measured on gfx950 with SQ_LDS_BANK_CONFLICT).
__device__ __forceinline__ int lds_swz(int row) { return (row >> 2) & 3; }
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * kRowBytes + ((chunk ^ lds_swz(row)) << 4);
}

// 16-bit K-contiguous tiles of BK K: rows of 2*BK bytes. The 16 lanes that
// serve one fragment read touch 16 consecutive rows at one logical chunk; the
// XOR spreads them over all 16 16-byte positions of a 256-byte bank window.
template <int BK>
__device__ __forceinline__ int swz_k(int row) {
  return BK == 32 ? (row >> 2) & 3 : (row >> 1) & 7;
}
template <int BK>
__device__ __forceinline__ int lds_off_k(int row, int chunk) {
  return row * (2 * BK) + ((chunk ^ swz_k<BK>(row)) << 4);
}

// XOR swizzle of the 16-byte chunks of a row-contiguous tile: the four K rows
// read by one 16-lane group of a transpose read land on distinct chunk
// positions (measured conflict-free).
__device__ __forceinline__ int swz_mn(int kr) { return (kr & 3) << 2; }

// Row permutation of fp32 row-contiguous tiles (register path): the
// transposing store writes 4 rows per thread; rotating rows by the thread's
// row block spreads one store instruction over distinct bank groups.
__device__ __forceinline__ int mn_row32(int r) { return r ^ ((r >> 2) & 3); }

__device__ __forceinline__ int xcd_remap(int bid, int n) {
  // Workgroups are dispatched round-robin over the 8 XCDs; give every XCD a
  // contiguous range of logical tiles so neighbours share its L2.
  const int x = bid & 7, idx = bid >> 3, per = n >> 3, rem = n & 7;
  return x * per + (x < rem ? x : rem) + idx;
}

// One operand restricted to the current output tile.
struct View {
  const uint8_t* p;   // element (tile row 0, k 0)
  int64_t ld_b;       // bytes between rows (k) or between K rows (mn)
  int64_t nrows;      // valid rows from tile row 0
  int64_t nk;         // valid K from k 0
};

// ---------------------------------------------------------------------------
// Contraction kinds. Operands 0..NA-1 are A (tile rows = output rows),
// NA..NA+NB-1 are B (tile rows = output columns); accumulator p multiplies
// A[pa(p)] by B[pb(p)]. Bit o of MN marks operand o as row-contiguous.
// WM x WN waves, each (32*MI) x (32*NI); NSTAGE LDS stages; DBUF: fragment
// registers double-buffered across K-substeps.
template <int NA_, int NB_, int NACC_, uint32_t MN_, int WM_, int WN_, int MI_, int NI_, int NSTAGE_,
          bool DBUF_, int BK_>
struct KindBase {
  static constexpr int NA = NA_, NB = NB_, NACC = NACC_, NOPS = NA_ + NB_;
  static constexpr uint32_t MN = MN_;
  static constexpr int WM = WM_, WN = WN_, MI = MI_, NI = NI_, NSTAGE = NSTAGE_;
  static constexpr bool DBUF = DBUF_;
  static constexpr int BK = BK_;             // K per LDS stage (16-bit path: 32 or 64)
  static_assert(BK == 32 || BK == 64, "K tile");
  static constexpr int THREADS = 64 * WM * WN;
  static constexpr int ROWS_A = 32 * MI * WM, ROWS_B = 32 * NI * WN;   // workgroup tile
  static constexpr bool is_mn(int o) { return (MN >> o) & 1u; }
  static constexpr int rows(int o) { return o < NA ? ROWS_A : ROWS_B; }
  // 16-bit stage layout: BK K x rows x 2 bytes per operand
  static constexpr int op_bytes(int o) { return rows(o) * BK * 2; }
  static constexpr int op_off(int o) {
    int s = 0;
    for (int i = 0; i < o; ++i) s += op_bytes(i);
    return s;
  }
  static constexpr int STAGE = op_off(NOPS);
  // which half of the block (threads 0-127 / 128-255) loads mn operand o (fp32 path)
  static constexpr int mn_half(int o) { return __builtin_popcount(MN & ((1u << o) - 1u)) & 1; }
};

#define LACT_KIND(NAME, NA, NB, NACC, MNMASK, WM, WN, MI, NI, NS, DBUF, BK, PA, PB) \
  struct NAME : KindBase<NA, NB, NACC, MNMASK, WM, WN, MI, NI, NS, DBUF, BK> {         \
    static constexpr int pa(int p) { return PA; }                                  \
    static constexpr int pb(int p) { return PB; }                                  \
  }

// 16-bit shapes: 8 waves (2 per SIMD); two-accumulator kinds use 64 x 64
// waves (128 x 256 tiles), one-accumulator kinds 128 x 64 (256 x 256).
// Kinds whose operands are all K-contiguous take 64 K per stage, so that every
// DMA fetches whole 128-byte lines; the gradient kinds (row-contiguous, 512
// bytes and more per K row) keep 32 K and twice the stages.
// Apply GEMM-1 and the key forward, hidden-major: A = W1, W3 (hidden rows),
// B = Q or K (token rows).
LACT_KIND(KApply16, 2, 1, 2, 0u, 2, 4, 2, 2, 2, true, 64, p, 0 * p);
// Hidden backward of the key forward: A = W2 read down its columns (hidden
// rows), B = V; accumulator D^T = (V W2)^T. Runs after KApply16 in the same
// workgroup, whose accumulators stay live.
LACT_KIND(KDual16, 1, 1, 1, 1u, 2, 4, 2, 2, 2, true, 64, 0 * p, 0 * p);
// Apply GEMM-2, feature-major: A = W2 (feature rows), B = hidden (token rows).
LACT_KIND(KOut16, 1, 1, 1, 0u, 2, 4, 4, 2, 2, true, 64, 0 * p, 0 * p);
// Gradients: A = eta dz1, eta dz3 (hidden rows), B = K (feature rows), all token-major.
LACT_KIND(KGrad13_16, 2, 1, 2, 7u, 2, 4, 2, 2, 4, true, 32, p, 0 * p);
// A = V (feature rows), B = eta hidden (hidden rows), token-major.
LACT_KIND(KGrad2_16, 1, 1, 1, 3u, 2, 4, 4, 2, 4, true, 32, 0 * p, 0 * p);
// Gradient with the weight update of whole rows (GRAD_UPD): A = eta dz1,
// eta dz3 or V (128 rows of W1, W3 or W2), B = K or eta hidden (every column,
// up to 512), token-major; waves of 64 x 128, 4 stages of 40 KiB.
LACT_KIND(KGradU16, 1, 1, 1, 3u, 2, 4, 2, 4, 4, true, 32, 0 * p, 0 * p);
// Narrow shapes (16-bit, d <= 128): the feature dimension fills 128 tile rows
// instead of half of 256. Apply GEMM-2: 128 features x 512 tokens; gradients
// of W1, W3: 256 hidden x 128 features; gradient of W2: 128 features x 256
// hidden.
LACT_KIND(KOutN16, 1, 1, 1, 0u, 2, 4, 2, 4, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KGrad13N16, 2, 1, 2, 7u, 4, 2, 2, 2, 4, true, 32, p, 0 * p);
LACT_KIND(KGrad2N16, 1, 1, 1, 3u, 2, 4, 2, 2, 4, true, 32, 0 * p, 0 * p);
// First launch for d <= 128 (16-bit): 4 waves of 64 x 64 (128 hidden x 128
// tokens) and three 32-K stages, so that a workgroup takes 72 KiB of LDS and
// two workgroups share a CU: with K = d this short, a
// tile's time is mostly the wait for its first stage and the epilogue, which
// the other workgroup's loop overlaps.
LACT_KIND(KApplyN16, 2, 1, 2, 0u, 2, 2, 2, 2, 3, true, 32, p, 0 * p);
LACT_KIND(KDualN16, 1, 1, 1, 1u, 2, 2, 2, 2, 3, true, 32, 0 * p, 0 * p);
// fp32 shapes: 4 waves of 64 x 64 (128 x 128 tiles), register path; the key
// forward and its hidden backward share one loop (A = W1, W3, W2; B = K, V).
LACT_KIND(KApply32, 2, 1, 2, 0u, 2, 2, 2, 2, 2, false, 32, p, 0 * p);
LACT_KIND(KUpdate32, 3, 2, 3, 1u << 2, 2, 2, 2, 2, 2, false, 32, p, (p == 2 ? 1 : 0));
LACT_KIND(KOut32, 1, 1, 1, 0u, 2, 2, 2, 2, 2, false, 32, 0 * p, 0 * p);
LACT_KIND(KGrad13_32, 2, 1, 2, 7u, 2, 2, 2, 2, 2, false, 32, p, 0 * p);
LACT_KIND(KGrad2_32, 1, 1, 1, 3u, 2, 2, 2, 2, 2, false, 32, 0 * p, 0 * p);
// Newton-Schulz products, each computed in the orientation whose transpose is
// stored (see k_ns): both operands K-contiguous (K), both row-contiguous (MN),
// or the first row-contiguous (TY: Y read down its columns). fp16 operands:
// 8 waves of 128 x 64 (256 x 256 tiles) for large Gram matrices, 4 waves of
// 64 x 64 (128 x 128) for small ones; fp32: 4 waves of 64 x 64.
LACT_KIND(KNsK16B, 1, 1, 1, 0u, 2, 4, 4, 2, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsMN16B, 1, 1, 1, 3u, 2, 4, 4, 2, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsTY16B, 1, 1, 1, 1u, 2, 4, 4, 2, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsK16S, 1, 1, 1, 0u, 2, 2, 2, 2, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsMN16S, 1, 1, 1, 3u, 2, 2, 2, 2, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsTY16S, 1, 1, 1, 1u, 2, 2, 2, 2, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsK32, 1, 1, 1, 0u, 2, 2, 2, 2, 2, false, 32, 0 * p, 0 * p);
// Last Newton-Schulz step with the weight update (k_ns_final): A = B (rows of
// the polynomial, K-contiguous), B = X4 read down its columns; 128 rows x up
// to 512 columns, waves of 64 x 128, 2 stages of 80 KiB.
LACT_KIND(KNsRow16, 1, 1, 1, 2u, 2, 4, 2, 4, 2, true, 64, 0 * p, 0 * p);
LACT_KIND(KNsMN32, 1, 1, 1, 3u, 2, 2, 2, 2, 2, false, 32, 0 * p, 0 * p);
LACT_KIND(KNsTY32, 1, 1, 1, 1u, 2, 2, 2, 2, 2, false, 32, 0 * p, 0 * p);
#undef LACT_KIND

template <typename T, bool BIG> struct NsKinds;
template <> struct NsKinds<_Float16, true> {
  using K = KNsK16B;
  using MN = KNsMN16B;
  using TY = KNsTY16B;
};
template <> struct NsKinds<_Float16, false> {
  using K = KNsK16S;
  using MN = KNsMN16S;
  using TY = KNsTY16S;
};
template <> struct NsKinds<float, false> {
  using K = KNsK32;
  using MN = KNsMN32;
  using TY = KNsTY32;
};

template <typename T> struct Kinds;
template <> struct Kinds<__bf16> {
  using Apply = KApply16;
  using Update = KApply16;   // followed by KDual16
  using Out = KOut16;
  using Grad13 = KGrad13_16;
  using Grad2 = KGrad2_16;
};
template <> struct Kinds<_Float16> {   // the backward of Newton-Schulz: fp16 operands
  using Apply = KApply16;
  using Update = KApply16;
  using Out = KOut16;
  using Grad13 = KGrad13_16;
  using Grad2 = KGrad2_16;
};
template <> struct Kinds<float> {
  using Apply = KApply32;
  using Update = KUpdate32;
  using Out = KOut32;
  using Grad13 = KGrad13_32;
  using Grad2 = KGrad2_32;
};

// Kinds of the first launch: apply, key forward and its hidden backward.
template <typename T, bool NARROW>
struct FwdKinds {
  using Apply = typename Kinds<T>::Apply;
  using Update = typename Kinds<T>::Update;
  using Dual = KDual16;
};
template <>
struct FwdKinds<__bf16, true> {
  using Apply = KApplyN16;
  using Update = KApplyN16;
  using Dual = KDualN16;
};

// Kinds of the second launch: the narrow shapes for 16-bit I/O with d <= 128.
template <typename T, bool NARROW>
struct BwdKinds {
  using Out = typename Kinds<T>::Out;
  using Grad13 = typename Kinds<T>::Grad13;
  using Grad2 = typename Kinds<T>::Grad2;
};
template <>
struct BwdKinds<__bf16, true> {
  using Out = KOutN16;
  using Grad13 = KGrad13N16;
  using Grad2 = KGrad2N16;
};
template <>
struct BwdKinds<_Float16, true> {   // the Newton-Schulz reverse's GRAD2 products on 128 x 256 tiles
  using Out = KOutN16;
  using Grad13 = KGrad13N16;
  using Grad2 = KGrad2N16;
};

template <class K>
using Acc = f32x16_t[K::NACC][K::MI][K::NI];

// Wave coordinates inside the workgroup and the epilogue map of accumulator
// register r of block (mi, ni) (32x32 MFMA output layout).
template <class K>
__device__ __forceinline__ int wave_m() { return (threadIdx.x >> 6) / K::WN; }
template <class K>
__device__ __forceinline__ int wave_n() { return (threadIdx.x >> 6) % K::WN; }
template <class K>
__device__ __forceinline__ int acc_row(int mi, int r) {
  const int lane = threadIdx.x & 63;
  return wave_m<K>() * 32 * K::MI + mi * 32 + ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3);
}
template <class K>
__device__ __forceinline__ int acc_col(int ni) {
  return wave_n<K>() * 32 * K::NI + ni * 32 + (threadIdx.x & 31);
}

// ===========================================================================
// fp32 register path (4 waves, 128 x 128, MI = NI = 2)

template <typename T>
__device__ __forceinline__ void gload_k(u32x4_t (&r)[4], const View& v, int64_t k0) {
  constexpr int E = Tr<T>::E;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = threadIdx.x + i * 256;
    const int row = q >> 2, c = q & 3;
    const int64_t k = k0 + c * E;
    u32x4_t x = {0u, 0u, 0u, 0u};
    if (row < v.nrows && k < v.nk)
      x = *reinterpret_cast<const u32x4_t*>(v.p + row * v.ld_b + k * (int64_t)sizeof(T));
    r[i] = x;
  }
}

__device__ __forceinline__ void sstore_k(uint8_t* tile, const u32x4_t (&r)[4]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = threadIdx.x + i * 256;
    *reinterpret_cast<u32x4_t*>(tile + lds_off(q >> 2, q & 3)) = r[i];
  }
}

template <typename T>
__device__ __forceinline__ void gload_mn(u32x4_t (&r)[4], const View& v, int64_t k0, int tt) {
  constexpr int E = Tr<T>::E, KG = Tr<T>::KG;
  const int kg = tt % KG, mb = tt / KG;
  const int row = mb * E;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t k = k0 + 4 * kg + i;
    u32x4_t x = {0u, 0u, 0u, 0u};
    if (row < v.nrows && k < v.nk)
      x = *reinterpret_cast<const u32x4_t*>(v.p + k * v.ld_b + row * (int64_t)sizeof(T));
    r[i] = x;
  }
}

// fp32: a thread holds 4 K rows x 4 elements; write 4 rows x 4 K.
__device__ __forceinline__ void sstore_mn32(uint8_t* tile, const u32x4_t (&r)[4], int tt) {
  const int kg = tt & 3, mb = tt >> 2;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int row = mn_row32(mb * 4 + m);
    *reinterpret_cast<u32x4_t*>(tile + lds_off(row, kg)) = u32x4_t{r[0][m], r[1][m], r[2][m], r[3][m]};
  }
}

__device__ __forceinline__ u32x4_t frag32(const uint8_t* tile, int row, int chunk, bool mn) {
  const int pr = mn ? mn_row32(row) : row;
  return *reinterpret_cast<const u32x4_t*>(tile + lds_off(pr, chunk));
}

template <class K>
__device__ __forceinline__ void compute_ktile32(const uint8_t* buf, Acc<K>& acc) {
  static_assert(K::MI == 2 && K::NI == 2 && K::THREADS == 256, "fp32 path shape");
  const int lane = threadIdx.x & 63;
  const int arow = wave_m<K>() * 64 + (lane & 31), brow = wave_n<K>() * 64 + (lane & 31);
  const int half = lane >> 5;
  // lanes 0-31 hold K 0..7 of the tile, lanes 32-63 K 8..15; MFMA s contracts
  // K s (first half-wave) and K 8+s (second half-wave)
  float af[K::NA][2][8], bf[K::NB][2][8];
#pragma unroll
  for (int o = 0; o < K::NA; ++o)
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
      // whole-vector bit casts: a bit cast of one vector element is not
      // reliable with this compiler (it reads element 0)
      const f32x4_t lo = __builtin_bit_cast(f32x4_t, frag32(buf + o * kTileBytes, arow + mi * 32, 2 * half, K::is_mn(o)));
      const f32x4_t hi =
          __builtin_bit_cast(f32x4_t, frag32(buf + o * kTileBytes, arow + mi * 32, 2 * half + 1, K::is_mn(o)));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        af[o][mi][e] = lo[e];
        af[o][mi][4 + e] = hi[e];
      }
    }
#pragma unroll
  for (int o = 0; o < K::NB; ++o)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const uint8_t* t = buf + (K::NA + o) * kTileBytes;
      const f32x4_t lo = __builtin_bit_cast(f32x4_t, frag32(t, brow + ni * 32, 2 * half, K::is_mn(K::NA + o)));
      const f32x4_t hi = __builtin_bit_cast(f32x4_t, frag32(t, brow + ni * 32, 2 * half + 1, K::is_mn(K::NA + o)));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bf[o][ni][e] = lo[e];
        bf[o][ni][4 + e] = hi[e];
      }
    }
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int p = 0; p < K::NACC; ++p)
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[p][mi][ni] =
              __builtin_amdgcn_mfma_f32_32x32x2f32(af[K::pa(p)][mi][s], bf[K::pb(p)][ni][s], acc[p][mi][ni], 0, 0, 0);
}

template <class K>
__device__ __forceinline__ void mainloop_regs(uint8_t* smem, const View (&ops)[K::NOPS], int64_t nk, Acc<K>& acc) {
  constexpr int BK = 16;
  const int nkt = (int)((nk + BK - 1) / BK);
  if (nkt <= 0) return;
  u32x4_t st[K::NOPS][4];
  auto gload = [&](int64_t k0) {
#pragma unroll
    for (int o = 0; o < K::NOPS; ++o) {
      if (K::is_mn(o)) {
        const int tt = threadIdx.x - 128 * K::mn_half(o);
        if (tt >= 0 && tt < 128) gload_mn<float>(st[o], ops[o], k0, tt);
      } else {
        gload_k<float>(st[o], ops[o], k0);
      }
    }
  };
  auto sstore = [&](uint8_t* buf) {
#pragma unroll
    for (int o = 0; o < K::NOPS; ++o) {
      if (K::is_mn(o)) {
        const int tt = threadIdx.x - 128 * K::mn_half(o);
        if (tt >= 0 && tt < 128) sstore_mn32(buf + o * kTileBytes, st[o], tt);
      } else {
        sstore_k(buf + o * kTileBytes, st[o]);
      }
    }
  };
  gload(0);
  sstore(smem);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const uint8_t* cur = smem + (kt & 1) * K::NOPS * kTileBytes;
    const bool more = kt + 1 < nkt;
    if (more) gload((int64_t)(kt + 1) * BK);
    compute_ktile32<K>(cur, acc);
    if (more) sstore(smem + ((kt + 1) & 1) * K::NOPS * kTileBytes);
    __syncthreads();
  }
}

// ===========================================================================
// 16-bit DMA path

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt_hi[15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
}

typedef __attribute__((address_space(3))) void lds_void_t;
__device__ __forceinline__ lds_void_t* to_lds(const void* p) { return (lds_void_t*)(p); }
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)to_lds(p); }

// Out-of-range buffer offset: the load returns zeros, so partial tiles arrive
// zero-padded in LDS.
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kRawBufferFlags = 0x00020000;

constexpr int kMaxSlots = 8;   // 16-byte DMA slots per lane and operand tile

// Slots: an operand tile of R rows and BK K is R*BK/8 slots of 16 bytes; lane
// `tid` of the workgroup fills slots tid, tid + THREADS, ... (so each wave
// instruction writes 1 KiB of consecutive LDS).
template <class K, int O>
struct Dma {
  static constexpr bool MN = K::is_mn(O);
  static constexpr int ROWS = K::rows(O);
  static constexpr int BK = K::BK;
  static constexpr int SLOTS = ROWS * BK / 8 / K::THREADS;   // per lane
  static_assert(SLOTS >= 1 && SLOTS <= kMaxSlots && ROWS * BK / 8 % K::THREADS == 0, "slot split");
  static constexpr int CPK = BK / 8;                          // chunks per row (k)
  static constexpr int CPR = ROWS / 8;                        // chunks per K row (mn)

  static __device__ __forceinline__ void offsets(uint32_t (&vo)[kMaxSlots], const View& v) {
#pragma unroll
    for (int i = 0; i < SLOTS; ++i) {
      const int p = i * K::THREADS + threadIdx.x;
      if (!MN) {
        const int row = p / CPK, c = (p % CPK) ^ swz_k<BK>(p / CPK);
        vo[i] = row < v.nrows ? (uint32_t)(row * v.ld_b + c * 16) : kOOB;
      } else {
        const int kr = p / CPR, c = (p % CPR) ^ swz_mn(p / CPR);
        vo[i] = c * 8 < v.nrows ? (uint32_t)(kr * v.ld_b + c * 16) : kOOB;
      }
    }
  }

  // DMA of k-tile kt into `tile`: a raw buffer descriptor whose base advances
  // with kt and whose size covers only the valid data, so K rows past the end
  // (row-contiguous operands) load as zeros. K-contiguous operands whose K is
  // not a multiple of BK zero the chunks past K in their last tile.
  static __device__ __forceinline__ void issue(uint8_t* tile, const View& v, const uint32_t (&vo)[kMaxSlots], int kt) {
    const uint8_t* base;
    int64_t span;
    if (!MN) {
      base = v.p + (int64_t)kt * BK * 2;
      const int64_t rows = v.nrows < ROWS ? v.nrows : ROWS;
      span = rows > 0 ? (rows - 1) * v.ld_b + BK * 2 : 0;
    } else {
      base = v.p + (int64_t)kt * BK * v.ld_b;
      int64_t rows = v.nk - (int64_t)kt * BK;
      rows = rows < 0 ? 0 : (rows > BK ? BK : rows);
      span = rows * v.ld_b;
    }
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)span, kRawBufferFlags);
    const int w = threadIdx.x >> 6;
    const int64_t kleft = v.nk - (int64_t)kt * BK;   // K left from this tile's start
#pragma unroll
    for (int i = 0; i < SLOTS; ++i) {
      uint32_t off = vo[i];
      if (!MN && kleft < BK) {
        const int p = i * K::THREADS + threadIdx.x;
        const int c = (p % CPK) ^ swz_k<BK>(p / CPK);
        if (c * 8 >= kleft) off = kOOB;
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, to_lds(tile + (i * K::THREADS + w * 64) * 16), 16, off, 0, 0,
                                               0);
    }
  }
};

// Every operand of kind K, unrolled at compile time.
template <class K, int O = 0>
struct DmaAll {
  static __device__ __forceinline__ void offsets(uint32_t (&vo)[K::NOPS][kMaxSlots], const View (&ops)[K::NOPS]) {
    if constexpr (O < K::NOPS) {
      Dma<K, O>::offsets(vo[O], ops[O]);
      DmaAll<K, O + 1>::offsets(vo, ops);
    }
  }
  static __device__ __forceinline__ void issue(uint8_t* st, const View (&ops)[K::NOPS],
                                               const uint32_t (&vo)[K::NOPS][kMaxSlots], int kt) {
    if constexpr (O < K::NOPS) {
      Dma<K, O>::issue(st + K::op_off(O), ops[O], vo[O], kt);
      DmaAll<K, O + 1>::issue(st, ops, vo, kt);
    }
  }
};

// LDS fragment reads are issued as inline asm, in program order, so that
// lgkmcnt can be counted exactly (wait for one substep's fragments while the
// next substep's reads are still in flight) and so that the compiler does not
// drain the in-flight DMA before them (it cannot tell which stage they touch).
__device__ __forceinline__ u32x4_t lds_read_b128(uint32_t a) {
  u32x4_t r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(a));
  return r;
}

// K-contiguous fragment: 8 K of row `row`, 16-byte chunk `chunk`.
template <int BK>
__device__ __forceinline__ u32x4_t frag_k(const uint8_t* tile, int row, int chunk) {
  return lds_read_b128(lds_addr(tile) + lds_off_k<BK>(row, chunk));
}

// Row-contiguous fragment (8 consecutive K of row rb + lane%32, K block
// 8*(lane/32) of substep s) by two transpose reads from a tile with `pitch`
// bytes per K row: within each 16-lane group source lane sl points at K row
// k0 + sl/4, columns 4*(sl%4)..+3, and output lane i receives column i, rows
// k0..k0+3.
__device__ __forceinline__ u32x4_t frag_tr(const uint8_t* tile, int rb, int s, int pitch) {
  const int lane = threadIdx.x & 63, g = lane >> 4, sl = lane & 15;
  const int mn = rb + 16 * (g & 1) + 4 * (sl & 3);
  const int c = mn >> 3, hb = (mn >> 2) & 1;
  const uint32_t base = lds_addr(tile);
  u32x2_t lo, hi;
  {
    const int kr = 16 * s + 8 * (g >> 1) + (sl >> 2);
    const uint32_t a = base + kr * pitch + ((c ^ swz_mn(kr)) << 4) + (hb << 3);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a));
  }
  {
    const int kr = 16 * s + 8 * (g >> 1) + 4 + (sl >> 2);
    const uint32_t a = base + kr * pitch + ((c ^ swz_mn(kr)) << 4) + (hb << 3);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(hi) : "v"(a));
  }
  return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
}

// Fragments of one K-substep (16 K) for this wave's tile.
template <class K>
struct Frags {
  u32x4_t a[K::NA][K::MI], b[K::NB][K::NI];
  // LDS instructions issued by load_frags (a transpose fragment takes two)
  static constexpr int kReads() {
    int n = 0;
    for (int o = 0; o < K::NOPS; ++o) n += (o < K::NA ? K::MI : K::NI) * (K::is_mn(o) ? 2 : 1);
    return n;
  }
};

template <class K>
__device__ __forceinline__ void load_frags(Frags<K>& f, const uint8_t* buf, int s) {
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int ab = wave_m<K>() * 32 * K::MI, bb = wave_n<K>() * 32 * K::NI;
#pragma unroll
  for (int o = 0; o < K::NA; ++o)
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi)
      f.a[o][mi] = K::is_mn(o) ? frag_tr(buf + K::op_off(o), ab + mi * 32, s, K::ROWS_A * 2)
                               : frag_k<K::BK>(buf + K::op_off(o), ab + mi * 32 + (lane & 31), 2 * s + half);
#pragma unroll
  for (int o = 0; o < K::NB; ++o)
#pragma unroll
    for (int ni = 0; ni < K::NI; ++ni)
      f.b[o][ni] = K::is_mn(K::NA + o) ? frag_tr(buf + K::op_off(K::NA + o), bb + ni * 32, s, K::ROWS_B * 2)
                                       : frag_k<K::BK>(buf + K::op_off(K::NA + o), bb + ni * 32 + (lane & 31),
                                                       2 * s + half);
}

// Wait until at most N LDS instructions are outstanding and make every
// fragment of f depend on that wait.
template <int N, class K>
__device__ __forceinline__ void frags_ready(Frags<K>& f) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(f.a[0][0]) : "n"(N));
#pragma unroll
  for (int o = 0; o < K::NA; ++o)
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi) asm volatile("" : "+v"(f.a[o][mi]));
#pragma unroll
  for (int o = 0; o < K::NB; ++o)
#pragma unroll
    for (int ni = 0; ni < K::NI; ++ni) asm volatile("" : "+v"(f.b[o][ni]));
}

template <typename T, class K>
__device__ __forceinline__ void mfma_frags(const Frags<K>& f, Acc<K>& acc) {
#pragma unroll
  for (int p = 0; p < K::NACC; ++p)
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < K::NI; ++ni) {
        if constexpr (__is_same(T, _Float16))
          acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
              __builtin_bit_cast(f16x8_t, f.a[K::pa(p)][mi]), __builtin_bit_cast(f16x8_t, f.b[K::pb(p)][ni]),
              acc[p][mi][ni], 0, 0, 0);
        else
          acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, f.a[K::pa(p)][mi]), __builtin_bit_cast(bf16x8_t, f.b[K::pb(p)][ni]),
              acc[p][mi][ni], 0, 0, 0);
      }
}

// NSTAGE k-tiles in flight, S = BK/16 MFMA substeps per tile. Per k-tile kt
// (stage kt % NS), with DBUF the fragment reads of substep s+1 are in flight
// while substep s multiplies; after the last reads of kt:
//   wait DMA of kt+1 | barrier | DMA kt+NS into the freed stage |
//   read substep 0 of kt+1 | MFMA substep S-1 of kt
// without DBUF every substep reads, waits and multiplies in turn.
// Hand-over of a free stage from one loop to the next one on the same LDS:
// in its last iteration a loop issues the first tile of the next loop into
// the stage it has just finished with, so the next loop starts with its first
// tile in flight instead of a cold prologue.
struct NoNext {
  __device__ __forceinline__ void first(int) {}
};
template <class K2, int SLOT>
struct ChainNext {
  uint8_t* smem;
  const View (&ops)[K2::NOPS];
  int slot;   // stage the first tile went to, -1 if none
  __device__ __forceinline__ ChainNext(uint8_t* s, const View (&o)[K2::NOPS]) : smem(s), ops(o), slot(-1) {}
  __device__ __forceinline__ void first(int s) {
    uint32_t vo[K2::NOPS][kMaxSlots];
    DmaAll<K2>::offsets(vo, ops);
    DmaAll<K2>::issue(smem + s * SLOT, ops, vo, 0);
    slot = s;
  }
};

// Stage t of this loop lives at smem + ((t + shift) % NSTAGE) * SLOT; with
// first_issued, tile 0 is already in flight there (issued by the previous
// loop's hand-over).
template <typename T, class K, int SLOT = K::STAGE, class Next = NoNext>
__device__ __forceinline__ void mainloop_dma(uint8_t* smem, const View (&ops)[K::NOPS], int64_t nk, Acc<K>& acc,
                                             int shift = 0, bool first_issued = false, Next* next = nullptr) {
  static_assert(SLOT >= K::STAGE, "stage slot");
  constexpr int BK = K::BK, NS = K::NSTAGE, S = BK / 16;
  constexpr int L = [] {          // DMA instructions per lane per k-tile
    int n = 0;
    for (int o = 0; o < K::NOPS; ++o) n += K::rows(o) * K::BK / 8 / K::THREADS;
    return n;
  }();
  constexpr int R = Frags<K>::kReads();
  static_assert(!K::DBUF || R < 16, "substep reads exceed lgkmcnt");
  static_assert(L * NS < 64, "DMA in flight exceeds vmcnt");
  static_assert(S % 2 == 0, "substeps per tile");
  const int nkt = (int)((nk + BK - 1) / BK);
  if (nkt <= 0) return;
  uint32_t vo[K::NOPS][kMaxSlots];
  DmaAll<K>::offsets(vo, ops);
  auto stage = [&](int kt) { return smem + ((kt + shift) % NS) * SLOT; };
  auto issue = [&](int kt) { DmaAll<K>::issue(stage(kt), ops, vo, kt); };
#pragma unroll
  for (int t = 0; t < NS; ++t)
    if (t < nkt && !(t == 0 && first_issued)) issue(t);
  if (nkt >= NS) wait_vmcnt<L * (NS - 1)>();
  else wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  if constexpr (K::DBUF) {
    Frags<K> f[2];
    load_frags<K>(f[0], stage(0), 0);
    for (int kt = 0; kt < nkt; ++kt) {
      const uint8_t* cur = stage(kt);
#pragma unroll
      for (int s = 0; s + 1 < S; ++s) {
        load_frags<K>(f[(s + 1) & 1], cur, s + 1);
        frags_ready<R, K>(f[s & 1]);           // substep s is in; s+1 still in flight
        mfma_frags<T, K>(f[s & 1], acc);
        __builtin_amdgcn_sched_barrier(0);     // issue all of them before the next wait
      }
      frags_ready<0, K>(f[(S - 1) & 1]);       // this wave is done reading tile kt
      if (kt + 1 < nkt) {
        if (kt + NS - 1 < nkt) wait_vmcnt<L * (NS - 2)>();   // tile kt+1 landed
        else wait_vmcnt<0>();
      }
      __builtin_amdgcn_s_barrier();            // every wave is past tile kt and has tile kt+1
      asm volatile("" ::: "memory");
      if (kt + NS < nkt) issue(kt + NS);       // refill the stage tile kt used
      else if (kt + NS == nkt && next) next->first((kt + shift) % NS);
      if (kt + 1 < nkt) load_frags<K>(f[0], stage(kt + 1), 0);
      mfma_frags<T, K>(f[(S - 1) & 1], acc);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    Frags<K> f;
    for (int kt = 0; kt < nkt; ++kt) {
      const uint8_t* cur = stage(kt);
#pragma unroll
      for (int s = 0; s < S; ++s) {
        load_frags<K>(f, cur, s);
        frags_ready<0, K>(f);
        mfma_frags<T, K>(f, acc);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (kt + 1 < nkt) {
        if (kt + NS - 1 < nkt) wait_vmcnt<L * (NS - 2)>();
        else wait_vmcnt<0>();
      }
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      if (kt + NS < nkt) issue(kt + NS);
      else if (kt + NS == nkt && next) next->first((kt + shift) % NS);
    }
  }
  // The caller may reuse LDS after the loop: every wave has waited for its
  // own LDS reads, and this loop's DMA has landed (the tail waits drain it).
  // A DMA handed over to the next loop keeps running: no vmcnt wait here.
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <class K>
__device__ __forceinline__ void zero_acc(Acc<K>& acc) {
#pragma unroll
  for (int p = 0; p < K::NACC; ++p)
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < K::NI; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[p][mi][ni][r] = 0.f;
}

// acc = sum over K of A[pa(p)] B[pb(p)]^T for this workgroup's tile.
template <typename T, class K>
__device__ __forceinline__ void mainloop(uint8_t* smem, const View (&ops)[K::NOPS], int64_t nk, Acc<K>& acc) {
  zero_acc<K>(acc);
  if constexpr (sizeof(T) == 2) mainloop_dma<T, K>(smem, ops, nk, acc);
  else mainloop_regs<K>(smem, ops, nk, acc);
}

// Two loops on one LDS ring of NSTAGE slots of SLOT bytes: the first hands
// its last free stage to the second (16-bit path).
template <typename T, class K1, class K2, int SLOT>
__device__ __forceinline__ void mainloop_chain(uint8_t* smem, const View (&ops1)[K1::NOPS], int64_t nk1, Acc<K1>& acc1,
                                               const View (&ops2)[K2::NOPS], int64_t nk2, Acc<K2>& acc2) {
  static_assert(sizeof(T) == 2 && K1::NSTAGE == K2::NSTAGE, "chained loops: 16-bit, one ring");
  zero_acc<K1>(acc1);
  zero_acc<K2>(acc2);
  ChainNext<K2, SLOT> nx(smem, ops2);
  mainloop_dma<T, K1, SLOT, ChainNext<K2, SLOT>>(smem, ops1, nk1, acc1, 0, false, &nx);
  mainloop_dma<T, K2, SLOT>(smem, ops2, nk2, acc2, nx.slot < 0 ? 0 : nx.slot, nx.slot >= 0);
}

template <typename T, class K>
constexpr int smem_bytes() {
  return sizeof(T) == 2 ? K::NSTAGE * K::STAGE : 2 * K::NOPS * kTileBytes;
}
constexpr int cmax(int a, int b) { return a > b ? a : b; }

// ===========================================================================
// Epilogue helpers

// Four consecutive elements (8 bytes of 16-bit or 16 bytes of fp32) at idx.
template <typename T>
__device__ __forceinline__ void st4(void* base, int64_t idx, float a, float b, float c, float d) {
  if constexpr (sizeof(T) == 2) {
    typedef __attribute__((ext_vector_type(4))) T t4;
    *reinterpret_cast<t4*>(reinterpret_cast<T*>(base) + idx) = t4{(T)a, (T)b, (T)c, (T)d};
  } else {
    *reinterpret_cast<float4*>(reinterpret_cast<float*>(base) + idx) = make_float4(a, b, c, d);
  }
}

__device__ __forceinline__ float sigmoidf_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

__device__ __forceinline__ View view_k(const Operand& op, int inst, int64_t row0, int64_t k0, int64_t nrows,
                                       int64_t nk, int esz) {
  const int64_t off = inst * op.inst_stride + row0 * op.ld + k0;
  return View{reinterpret_cast<const uint8_t*>(op.base) + off * esz, op.ld * esz, nrows, nk};
}
__device__ __forceinline__ View view_mn(const Operand& op, int inst, int64_t row0, int64_t k0, int64_t nrows,
                                        int64_t nk, int esz) {
  const int64_t off = inst * op.inst_stride + k0 * op.ld + row0;
  return View{reinterpret_cast<const uint8_t*>(op.base) + off * esz, op.ld * esz, nrows, nk};
}

// Workgroup barrier for LDS hand-offs only: waits for this wave's LDS
// operations, not for its global stores (which __syncthreads would drain).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Output staging (16-bit): an accumulator tile of R output rows (hidden units
// or features, the MFMA row index) x C tokens is written to LDS token-major,
// R*2 bytes per token row, and then copied to the token-major output with
// 16-byte lanes, 16 or 32 lanes per token row: every store instruction writes
// whole 128-byte lines instead of 16-byte pieces of 32 lines. The 16-byte
// chunks of a row are XOR-rotated by the token's low 4 bits, so that the 32
// tokens of one accumulator write and the 16 chunks of one row read spread
// over all banks.
template <int R, typename E = __bf16>
__device__ __forceinline__ void stage_put(uint8_t* buf, int tok, int row, float a, float b, float c, float d) {
  typedef __attribute__((ext_vector_type(4))) E e4_t;
  const int off = tok * (2 * R) + ((((row >> 3) ^ (tok & 15))) << 4) + (((row >> 2) & 1) << 3);
  *reinterpret_cast<e4_t*>(buf + off) = e4_t{(E)a, (E)b, (E)c, (E)d};
}

// Copy the staged tile to out (element (token 0, row 0) of the tile, ld
// elements between tokens): tokens < ntok, rows < nrow (a multiple of 8).
template <int R, int C, int THREADS, typename E = __bf16>
__device__ __forceinline__ void stage_flush(const uint8_t* buf, E* out, int64_t ld, int64_t ntok, int64_t nrow) {
  constexpr int CPR = R / 8, TOTAL = C * CPR;
  static_assert(CPR >= 16 && TOTAL % THREADS == 0, "staging shape");
#pragma unroll
  for (int i = 0; i < TOTAL / THREADS; ++i) {
    const int q = i * THREADS + threadIdx.x;
    const int tok = q / CPR, c = q % CPR;
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(buf + tok * (2 * R) + ((c ^ (tok & 15)) << 4));
    if (tok < ntok && c * 8 < nrow) *reinterpret_cast<u32x4_t*>(out + tok * ld + c * 8) = v;
  }
}

// Key-forward epilogue: from Z1, Z3 and D = W2^T v (hidden-major tiles) write
// eta*hidden, eta*dz1 and eta*dz3 token-major, four hidden units per store.
// With per-matrix rates (lr1, lr2, lr3) per token, hidden (the W2 gradient)
// takes lr2, dz1 (W1) lr1 and dz3 (W3) lr3 (Alg. 1, update).
template <typename T, class K, bool KEEP = false>
__device__ __forceinline__ void update_epilogue(const f32x16_t (&z1a)[K::MI][K::NI], const f32x16_t (&z3a)[K::MI][K::NI],
                                                const f32x16_t (&dda)[K::MI][K::NI], const FwdSeg& sg, int inst,
                                                int64_t j0, int64_t i0, int64_t hrows, int64_t ntok, int h) {
  const int lane = threadIdx.x & 63;
  const int64_t ob = inst * sg.out_inst;
  const int es = sg.eta_stride, o2 = es > 1 ? 1 : 0;
  const float* eta = sg.eta + inst * sg.eta_inst + i0 * es;
  const int hrow0 = wave_m<K>() * 32 * K::MI + ((lane >> 5) << 2);
#pragma unroll
  for (int ni = 0; ni < K::NI; ++ni) {
    const int tok = acc_col<K>(ni);
    if (tok >= ntok) continue;
    const float e1 = eta[tok * es], e2 = eta[tok * es + o2], e3 = eta[tok * es + 2 * o2];
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int hid = hrow0 + mi * 32 + 8 * g;
        if (hid >= hrows) continue;
        float vh[4], vg[4], vb[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          const float z1 = z1a[mi][ni][r], z3 = z3a[mi][ni][r], dh = dda[mi][ni][r];
          const float s = sigmoidf_fast(z1);
          const float a = z1 * s;                     // SiLU(z1)
          vh[e] = e2 * a * z3;                        // eta * hidden
          vg[e] = e1 * dh * z3 * s * (1.0f + z1 * (1.0f - s));   // eta * dz1
          vb[e] = e3 * dh * a;                        // eta * dz3
        }
        const int64_t idx = ob + (i0 + tok) * h + j0 + hid;
        st4<T>(sg.out1, idx, vh[0], vh[1], vh[2], vh[3]);
        st4<T>(sg.out2, idx, vg[0], vg[1], vg[2], vg[3]);
        st4<T>(sg.out3, idx, vb[0], vb[1], vb[2], vb[3]);
        if constexpr (KEEP) {
          const int64_t kx = inst * sg.keep_inst + (i0 + tok) * h + j0 + hid;
          const int r = 4 * g;
          st4<T>(sg.keep[0], kx, z1a[mi][ni][r], z1a[mi][ni][r + 1], z1a[mi][ni][r + 2], z1a[mi][ni][r + 3]);
          st4<T>(sg.keep[1], kx, z3a[mi][ni][r], z3a[mi][ni][r + 1], z3a[mi][ni][r + 2], z3a[mi][ni][r + 3]);
          st4<T>(sg.keep[2], kx, dda[mi][ni][r], dda[mi][ni][r + 1], dda[mi][ni][r + 2], dda[mi][ni][r + 3]);
        }
      }
  }
}

// The same for 16-bit outputs, staged through LDS (two 64 KiB buffers):
// eta*hidden and eta*dz1 first, then eta*dz3.
template <class K, bool KEEP = false>
__device__ __forceinline__ void update_epilogue_staged(const f32x16_t (&z1a)[K::MI][K::NI],
                                                       const f32x16_t (&z3a)[K::MI][K::NI],
                                                       const f32x16_t (&dda)[K::MI][K::NI], const FwdSeg& sg,
                                                       int inst, int64_t j0, int64_t i0, int64_t hrows,
                                                       int64_t ntok, int h, uint8_t* smem) {
  constexpr int R = K::ROWS_A, C = K::ROWS_B;
  uint8_t* buf0 = smem;
  uint8_t* buf1 = smem + R * C * 2;
  const int lane = threadIdx.x & 63;
  const int es = sg.eta_stride, o2 = es > 1 ? 1 : 0;
  const float* eta = sg.eta + inst * sg.eta_inst + i0 * es;
  const int hrow0 = wave_m<K>() * 32 * K::MI + ((lane >> 5) << 2);
  float e1[K::NI], e2[K::NI], e3[K::NI];   // rates of dz1 (W1), hidden (W2), dz3 (W3)
#pragma unroll
  for (int ni = 0; ni < K::NI; ++ni) {
    const int tok = acc_col<K>(ni);
    const bool in = tok < ntok;
    e1[ni] = in ? eta[tok * es] : 0.0f;
    e2[ni] = in ? eta[tok * es + o2] : 0.0f;
    e3[ni] = in ? eta[tok * es + 2 * o2] : 0.0f;
  }
  if constexpr (KEEP) {   // Z1 and Z3, then D, for the backward's reverse of this update (first:
                           // every accumulator is live here anyway)
    const int64_t kt = inst * sg.keep_inst + i0 * h + j0;
#pragma unroll
    for (int ni = 0; ni < K::NI; ++ni)
#pragma unroll
      for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int tok = acc_col<K>(ni), row = hrow0 + mi * 32 + 8 * g, r = 4 * g;
          stage_put<R>(buf0, tok, row, z1a[mi][ni][r], z1a[mi][ni][r + 1], z1a[mi][ni][r + 2], z1a[mi][ni][r + 3]);
          stage_put<R>(buf1, tok, row, z3a[mi][ni][r], z3a[mi][ni][r + 1], z3a[mi][ni][r + 2], z3a[mi][ni][r + 3]);
        }
    lds_barrier();
    stage_flush<R, C, K::THREADS>(buf0, reinterpret_cast<__bf16*>(sg.keep[0]) + kt, h, ntok, hrows);
    stage_flush<R, C, K::THREADS>(buf1, reinterpret_cast<__bf16*>(sg.keep[1]) + kt, h, ntok, hrows);
    lds_barrier();
#pragma unroll
    for (int ni = 0; ni < K::NI; ++ni)
#pragma unroll
      for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = 4 * g;
          stage_put<R>(buf0, acc_col<K>(ni), hrow0 + mi * 32 + 8 * g, dda[mi][ni][r], dda[mi][ni][r + 1],
                       dda[mi][ni][r + 2], dda[mi][ni][r + 3]);
        }
    lds_barrier();
    stage_flush<R, C, K::THREADS>(buf0, reinterpret_cast<__bf16*>(sg.keep[2]) + kt, h, ntok, hrows);
    lds_barrier();
  }
#pragma unroll
  for (int ni = 0; ni < K::NI; ++ni)
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float vh[4], vg[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          const float z1 = z1a[mi][ni][r], z3 = z3a[mi][ni][r];
          const float s = sigmoidf_fast(z1);
          vh[e] = e2[ni] * z1 * s * z3;
          vg[e] = e1[ni] * dda[mi][ni][r] * z3 * s * (1.0f + z1 * (1.0f - s));
        }
        const int tok = acc_col<K>(ni), row = hrow0 + mi * 32 + 8 * g;
        stage_put<R>(buf0, tok, row, vh[0], vh[1], vh[2], vh[3]);
        stage_put<R>(buf1, tok, row, vg[0], vg[1], vg[2], vg[3]);
      }
  lds_barrier();
  const int64_t tile = inst * sg.out_inst + i0 * h + j0;
  stage_flush<R, C, K::THREADS>(buf0, reinterpret_cast<__bf16*>(sg.out1) + tile, h, ntok, hrows);
  stage_flush<R, C, K::THREADS>(buf1, reinterpret_cast<__bf16*>(sg.out2) + tile, h, ntok, hrows);
  lds_barrier();
#pragma unroll
  for (int ni = 0; ni < K::NI; ++ni)
#pragma unroll
    for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float vb[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          const float z1 = z1a[mi][ni][r];
          vb[e] = e3[ni] * dda[mi][ni][r] * z1 * sigmoidf_fast(z1);
        }
        stage_put<R>(buf0, acc_col<K>(ni), hrow0 + mi * 32 + 8 * g, vb[0], vb[1], vb[2], vb[3]);
      }
  lds_barrier();
  stage_flush<R, C, K::THREADS>(buf0, reinterpret_cast<__bf16*>(sg.out3) + tile, h, ntok, hrows);
}

// ===========================================================================
// First launch of a chunk. Accumulators are hidden-major (rows = hidden units
// j, columns = tokens i): every lane holds four consecutive hidden units of
// one token per register group, written as one packed store into the
// token-major [tokens x h] output.
template <typename T, bool NARROW>
constexpr int fwd_smem() {
  using FK = FwdKinds<T, NARROW>;
  using KU = typename FK::Update;
  return cmax(smem_bytes<T, typename FK::Apply>(),
              cmax(smem_bytes<T, KU>(), sizeof(T) == 2 ? cmax(smem_bytes<T, typename FK::Dual>(),
                                                              2 * KU::ROWS_A * KU::ROWS_B * 2)
                                                       : 0));
}

template <typename T, bool NARROW, bool KEEP = false>
__device__ __forceinline__ void fwd_body(const FwdArgs& args, uint8_t* smem) {
  using KA = typename FwdKinds<T, NARROW>::Apply;
  using KU = typename FwdKinds<T, NARROW>::Update;
  static_assert(KA::THREADS == KU::THREADS, "one block size per launch");
  constexpr int kSmem = fwd_smem<T, NARROW>();
  constexpr int esz = sizeof(T);
  int bid = blockIdx.x;
  const bool first = bid < args.seg[0].nblocks;
  const FwdSeg& sg = first ? args.seg[0] : args.seg[1];
  if (!first) bid -= args.seg[0].nblocks;
  bid = xcd_remap(bid, sg.nblocks);   // per segment: every XCD gets a share of each kind
  const int per = sg.tiles_m * sg.tiles_n;
  const int inst = bid / per;
  const int rr = bid - inst * per;
  const int d = args.d, h = args.h;
  const int lane = threadIdx.x & 63;

  if (sg.kind == FWD_APPLY) {
    const int64_t j0 = (int64_t)(rr % sg.tiles_m) * KA::ROWS_A;   // hidden tile (fastest)
    const int64_t i0 = (int64_t)(rr / sg.tiles_m) * KA::ROWS_B;   // token tile
    const int64_t hrows = h - j0, ntok = sg.rows - i0;
    const View ops[3] = {view_k(args.w1, inst, j0, 0, hrows, d, esz), view_k(args.w3, inst, j0, 0, hrows, d, esz),
                         view_k(sg.a0, inst, i0, 0, ntok, d, esz)};
    Acc<KA> acc;
    mainloop<T, KA>(smem, ops, d, acc);
    void* out = reinterpret_cast<uint8_t*>(sg.out0) + (inst * sg.out_inst) * esz;
    const int hrow0 = wave_m<KA>() * 32 * KA::MI + ((lane >> 5) << 2);
    if constexpr (sizeof(T) == 2) {
      static_assert(KA::ROWS_A * KA::ROWS_B * 2 <= kSmem, "staging fits");
#pragma unroll
      for (int ni = 0; ni < KA::NI; ++ni)
#pragma unroll
        for (int mi = 0; mi < KA::MI; ++mi)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float z1 = acc[0][mi][ni][4 * g + e], z3 = acc[1][mi][ni][4 * g + e];
              v[e] = z1 * sigmoidf_fast(z1) * z3;
            }
            stage_put<KA::ROWS_A>(smem, acc_col<KA>(ni), hrow0 + mi * 32 + 8 * g, v[0], v[1], v[2], v[3]);
          }
      lds_barrier();
      stage_flush<KA::ROWS_A, KA::ROWS_B, KA::THREADS>(smem, reinterpret_cast<__bf16*>(out) + i0 * h + j0, h, ntok,
                                                         hrows);
      return;
    }
#pragma unroll
    for (int ni = 0; ni < KA::NI; ++ni) {
      const int tok = acc_col<KA>(ni);
      if (tok >= ntok) continue;
#pragma unroll
      for (int mi = 0; mi < KA::MI; ++mi)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int hid = hrow0 + mi * 32 + 8 * g;
          if (hid >= hrows) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float z1 = acc[0][mi][ni][4 * g + e], z3 = acc[1][mi][ni][4 * g + e];
            v[e] = z1 * sigmoidf_fast(z1) * z3;
          }
          st4<T>(out, (i0 + tok) * h + j0 + hid, v[0], v[1], v[2], v[3]);
        }
    }
  } else {
    const int64_t j0 = (int64_t)(rr % sg.tiles_m) * KU::ROWS_A;
    const int64_t i0 = (int64_t)(rr / sg.tiles_m) * KU::ROWS_B;
    const int64_t hrows = h - j0, ntok = sg.rows - i0;
    const View w1 = view_k(args.w1, inst, j0, 0, hrows, d, esz), w3 = view_k(args.w3, inst, j0, 0, hrows, d, esz);
    const View w2 = view_mn(args.w2, inst, j0, 0, hrows, d, esz);
    const View kk = view_k(sg.a0, inst, i0, 0, ntok, d, esz), vv = view_k(sg.a1, inst, i0, 0, ntok, d, esz);
    if constexpr (sizeof(T) == 2) {
      // Z1^T, Z3^T first, then D^T with the Z accumulators held: one
      // accumulator set per loop keeps the loops free of register spills.
      using KD = typename FwdKinds<T, NARROW>::Dual;
      static_assert(KD::ROWS_A == KU::ROWS_A && KD::ROWS_B == KU::ROWS_B && KD::WM == KU::WM &&
                        KD::MI == KU::MI && KD::NI == KU::NI, "accumulator layouts match");
      Acc<KU> az;
      Acc<KD> ad;
      const View opz[3] = {w1, w3, kk};
      const View opd[2] = {w2, vv};
      constexpr int kSlot = KU::STAGE > KD::STAGE ? KU::STAGE : KD::STAGE;
      static_assert(KU::NSTAGE * kSlot <= kSmem, "chained ring fits");
      mainloop_chain<T, KU, KD, kSlot>(smem, opz, d, az, opd, d, ad);
      static_assert(2 * KU::ROWS_A * KU::ROWS_B * 2 <= kSmem, "staging fits");
      update_epilogue_staged<KU, KEEP>(az[0], az[1], ad[0], sg, inst, j0, i0, hrows, ntok, h, smem);
    } else {
      const View ops[5] = {w1, w3, w2, kk, vv};
      Acc<KU> acc;
      mainloop<T, KU>(smem, ops, d, acc);
      update_epilogue<T, KU, KEEP>(acc[0], acc[1], acc[2], sg, inst, j0, i0, hrows, ntok, h);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(Kinds<T>::Apply::THREADS) void k_fwd(const FwdArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[fwd_smem<T, false>()];
  fwd_body<T, false>(args, smem);
}

// d <= 128, 16-bit: two workgroups per CU (at most 256 VGPRs per wave).
__global__ __launch_bounds__(KApplyN16::THREADS) __attribute__((amdgpu_waves_per_eu(2))) void k_fwd_narrow(
    const FwdArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[fwd_smem<__bf16, true>()];
  fwd_body<__bf16, true>(args, smem);
}

// The same two kernels with the key forward's Z1, Z3 and D written out too
// (FwdSeg::keep): the backward's replay of an update, whose reverse reads
// them instead of computing the three products again.
template <typename T>
__global__ __launch_bounds__(Kinds<T>::Apply::THREADS) void k_fwd_keep(const FwdArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[fwd_smem<T, false>()];
  fwd_body<T, false, true>(args, smem);
}

__global__ __launch_bounds__(KApplyN16::THREADS) __attribute__((amdgpu_waves_per_eu(2))) void k_fwd_narrow_keep(
    const FwdArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[fwd_smem<__bf16, true>()];
  fwd_body<__bf16, true, true>(args, smem);
}

// The weight update of a GRAD_UPD tile from its accumulators P (= -g):
//   U = W + P,  W <- U ||W_row|| / ||U_row||   (§3.2 weight normalisation; Alg. 1)
// or, with momentum (App. A; Table 3), Y = P - bbar M, M <- -Y, U = W + Y;
// with ADD (the last Newton-Schulz step) the step is P + xa X, X in W's layout.
// The tile goes through LDS in passes of RP rows, so that lanes stream W (and
// M) along whole rows in 16-byte vectors, as the separate update kernel does:
// the rows of a pass are staged by the waves that hold them, TPR lanes share a
// row, and a row's squared norms are summed over those lanes by shuffles. A
// pass issues its W (and M) loads before the hand-over through LDS.
template <class KG, bool MOM, bool ADD = false>
__device__ __forceinline__ void update_rows(Acc<KG>& acc, float* W, __bf16* Wb, float* M, float bb, int64_t mrows,
                                            int cols, uint8_t* smem, const float* X = nullptr, float xa = 0.f) {
  static_assert(!(MOM && ADD), "one extra operand");
  constexpr int RP = (MOM || ADD) ? 32 : 64;       // rows per pass
  constexpr int TPR = KG::THREADS / RP;             // lanes per row
  constexpr int NV = KG::ROWS_B / 4 / TPR;          // 16-byte vectors per lane
  constexpr int PITCH = KG::ROWS_B + 4;             // floats per LDS row
  static_assert(KG::NACC == 1 && TPR <= 64 && RP * PITCH * 4 <= KG::NSTAGE * KG::STAGE, "update passes");
  typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4_t;
  float* st = reinterpret_cast<float*>(smem);
  const int lr = threadIdx.x / TPR, part = threadIdx.x % TPR;
  const int nv = cols >> 2;
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int pass = 0; pass < KG::ROWS_A / RP; ++pass) {
    const int64_t row = (int64_t)pass * RP + lr;
    const bool rok = row < mrows;
    float4 w[NV], m[(MOM || ADD) ? NV : 1];
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int c4 = part + TPR * q;
      const bool ok = rok && c4 < nv;
      w[q] = ok ? reinterpret_cast<const float4*>(W + row * cols)[c4] : zero;
      if constexpr (MOM) m[q] = ok ? reinterpret_cast<const float4*>(M + row * cols)[c4] : zero;
      if constexpr (ADD) m[q] = ok ? reinterpret_cast<const float4*>(X + row * cols)[c4] : zero;
    }
    // stage the accumulator rows [pass*RP, pass*RP + RP) (32-row blocks mi of wave row wave_m)
#pragma unroll
    for (int mi = 0; mi < KG::MI; ++mi) {
      const int blk = wave_m<KG>() * 32 * KG::MI + mi * 32;
      if (blk >= pass * RP && blk < pass * RP + RP) {
#pragma unroll
        for (int ni = 0; ni < KG::NI; ++ni)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            st[(acc_row<KG>(mi, r) - pass * RP) * PITCH + acc_col<KG>(ni)] = acc[0][mi][ni][r];
      }
    }
    lds_barrier();
    float su = 0.f, sw = 0.f;
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      float4 y = reinterpret_cast<const float4*>(st + lr * PITCH)[part + TPR * q];
      if constexpr (MOM) {
        y = make_float4(fmaf(-bb, m[q].x, y.x), fmaf(-bb, m[q].y, y.y), fmaf(-bb, m[q].z, y.z),
                        fmaf(-bb, m[q].w, y.w));
        m[q] = make_float4(-y.x, -y.y, -y.z, -y.w);
      }
      if constexpr (ADD)
        y = make_float4(fmaf(xa, m[q].x, y.x), fmaf(xa, m[q].y, y.y), fmaf(xa, m[q].z, y.z), fmaf(xa, m[q].w, y.w));
      const float4 x = w[q];
      sw += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
      w[q] = make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
      su += w[q].x * w[q].x + w[q].y * w[q].y + w[q].z * w[q].z + w[q].w * w[q].w;
    }
#pragma unroll
    for (int off = 1; off < TPR; off <<= 1) {
      su += __shfl_xor(su, off, TPR);
      sw += __shfl_xor(sw, off, TPR);
    }
    const float f = sqrtf(sw) / sqrtf(su);
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int c4 = part + TPR * q;
      if (rok && c4 < nv) {
        const float4 x = make_float4(w[q].x * f, w[q].y * f, w[q].z * f, w[q].w * f);
        reinterpret_cast<float4*>(W + row * cols)[c4] = x;
        reinterpret_cast<bf16x4_t*>(Wb + row * cols)[c4] = bf16x4_t{(__bf16)x.x, (__bf16)x.y, (__bf16)x.z, (__bf16)x.w};
        if constexpr (MOM) reinterpret_cast<float4*>(M + row * cols)[c4] = m[q];
      }
    }
    if (pass + 1 < KG::ROWS_A / RP) lds_barrier();   // the pass is read before the next is staged
  }
}

// GRAD_UPD tile (16-bit operands): 128 rows of W1, W3 or W2 with all their
// columns. The chunk's tokens are contracted into P = -g in fp32 registers
// (P1 = (eta dz1)^T K, P3 = (eta dz3)^T K, P2 = V^T (eta hidden)); then the
// weight update of the same rows (update_rows), in place on the fp32 state
// (and the momentum state), with the bf16 operand copy of the result for the
// next chunk.
template <typename T>
__device__ __forceinline__ void grad_update_tile(const BwdSeg& sg, int inst, int rr, int d, int h, uint8_t* smem) {
  using KG = KGradU16;
  const int t1 = (h + KG::ROWS_A - 1) / KG::ROWS_A;   // row tiles of W1 (and of W3)
  int mat, tile;
  if (rr < t1) {
    mat = 0;
    tile = rr;
  } else if (rr < 2 * t1) {
    mat = 2;
    tile = rr - t1;
  } else {
    mat = 1;
    tile = rr - 2 * t1;
  }
  const int cols = mat == 1 ? h : d;
  const int64_t r0 = (int64_t)tile * KG::ROWS_A;
  const int64_t mrows = (mat == 1 ? d : h) - r0;
  const Operand& A = mat == 0 ? sg.a0 : (mat == 2 ? sg.a1 : sg.a2);
  const Operand& B = mat == 1 ? sg.b1 : sg.b0;
  const View ops[2] = {view_mn(A, inst, r0, 0, mrows, sg.rows, 2), view_mn(B, inst, 0, 0, cols, sg.rows, 2)};
  Acc<KG> acc;
  mainloop<T, KG>(smem, ops, sg.rows, acc);

  const int64_t dh = (int64_t)d * h;
  const int64_t base = inst * dh + r0 * cols;
  if (sg.M[0]) update_rows<KG, true>(acc, sg.W[mat] + base, reinterpret_cast<__bf16*>(sg.Wb[mat]) + base,
                                     sg.M[mat] + base, sg.bbar[(int64_t)inst * sg.bbar_stride], mrows, cols, smem);
  else update_rows<KG, false>(acc, sg.W[mat] + base, reinterpret_cast<__bf16*>(sg.Wb[mat]) + base, nullptr, 0.f,
                              mrows, cols, smem);
}

// Sums of squares of accumulators 0 and NACC-1 of this workgroup's tile (for
// the Frobenius norm of the gradient that Newton-Schulz divides by), in
// thread 0; reuses the start of LDS, which the caller has finished with.
template <class K>
__device__ __forceinline__ float2 tile_sumsq(const Acc<K>& acc, uint8_t* smem) {
  float a = 0.f, b = 0.f;
#pragma unroll
  for (int mi = 0; mi < K::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < K::NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        a = fmaf(acc[0][mi][ni][r], acc[0][mi][ni][r], a);
        b = fmaf(acc[K::NACC - 1][mi][ni][r], acc[K::NACC - 1][mi][ni][r], b);
      }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
  }
  float* red = reinterpret_cast<float*>(smem);
  constexpr int NW = K::THREADS / 64;
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = a;
    red[NW + (threadIdx.x >> 6)] = b;
  }
  lds_barrier();
  float2 t = make_float2(0.f, 0.f);
  if (threadIdx.x == 0)
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      t.x += red[w];
      t.y += red[NW + w];
    }
  return t;
}

// Second launch: apply GEMM-2 and the gradient contractions (split over tokens).
template <typename T, bool NARROW>
constexpr int bwd_smem() {
  using KO = typename BwdKinds<T, NARROW>::Out;
  using K13 = typename BwdKinds<T, NARROW>::Grad13;
  using K2 = typename BwdKinds<T, NARROW>::Grad2;
  return cmax(cmax(smem_bytes<T, KO>(), (sizeof(T) == 2 && !NARROW) ? smem_bytes<T, KGradU16>() : 0),
              cmax(smem_bytes<T, K13>(), smem_bytes<T, K2>()));
}

// Block `blk` of the second launch (smem: bwd_smem bytes of LDS).
template <typename T, bool NARROW>
__device__ __forceinline__ void bwd_body(const BwdArgs& args, int blk, uint8_t* smem) {
  using KO = typename BwdKinds<T, NARROW>::Out;
  using K13 = typename BwdKinds<T, NARROW>::Grad13;
  using K2 = typename BwdKinds<T, NARROW>::Grad2;
  static_assert(KO::THREADS == K13::THREADS && KO::THREADS == K2::THREADS, "one block size per launch");
  constexpr int esz = sizeof(T);
  int bid = blk;
  int si = 0;
  while (si + 1 < args.nseg && bid >= args.seg[si].nblocks) {
    bid -= args.seg[si].nblocks;
    ++si;
  }
  const BwdSeg& sg = args.seg[si];
  bid = xcd_remap(bid, sg.nblocks);
  const int d = args.d, h = args.h;
  const int per = sg.tiles_m * sg.tiles_n;
  const int per_inst = per * sg.nsplit;
  const int inst = bid / per_inst;
  int rr = bid - inst * per_inst;
  const int split = rr / per;
  rr -= split * per;
  const int lane = threadIdx.x & 63;

  if (sg.kind == BWD_OUT) {
    // O^T[m, i] = sum_j W2[m, j] hidden[i, j]: feature-major accumulators, four
    // consecutive features of one token per register group -> packed stores
    const int64_t m0 = (int64_t)(rr % sg.tiles_m) * KO::ROWS_A;   // feature tile (fastest)
    const int64_t t0 = (int64_t)(rr / sg.tiles_m) * KO::ROWS_B;   // token tile
    const int64_t mrows = d - m0, ntok = sg.rows - t0;
    const int64_t kk = sg.klen ? sg.klen : h;   // contraction length of this segment
    const View ops[2] = {view_k(sg.b0, inst, m0, 0, mrows, kk, esz), view_k(sg.a0, inst, t0, 0, ntok, kk, esz)};
    Acc<KO> acc;
    mainloop<T, KO>(smem, ops, kk, acc);
    const int64_t ob = inst * sg.out_inst;
    const int mrow0 = wave_m<KO>() * 32 * KO::MI + ((lane >> 5) << 2);
    if (sg.row_scale) {   // per-token factor of the output rows
#pragma unroll
      for (int ni = 0; ni < KO::NI; ++ni) {
        const int tok = acc_col<KO>(ni);
        const float sc = tok < ntok ? sg.row_scale[inst * sg.scale_inst + t0 + tok] : 0.0f;
#pragma unroll
        for (int mi = 0; mi < KO::MI; ++mi)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[0][mi][ni][r] *= sc;
      }
    }
    if constexpr (sizeof(T) == 2) {
      static_assert(KO::ROWS_A * KO::ROWS_B * 2 <= bwd_smem<T, NARROW>(), "staging fits");
#pragma unroll
      for (int ni = 0; ni < KO::NI; ++ni)
#pragma unroll
        for (int mi = 0; mi < KO::MI; ++mi)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x16_t& a = acc[0][mi][ni];
            stage_put<KO::ROWS_A, T>(smem, acc_col<KO>(ni), mrow0 + mi * 32 + 8 * g, a[4 * g], a[4 * g + 1],
                                  a[4 * g + 2], a[4 * g + 3]);
          }
      lds_barrier();
      stage_flush<KO::ROWS_A, KO::ROWS_B, KO::THREADS, T>(smem, reinterpret_cast<T*>(sg.out) + ob + t0 * d + m0, d,
                                                         ntok, mrows);
      return;
    }
#pragma unroll
    for (int ni = 0; ni < KO::NI; ++ni) {
      const int tok = acc_col<KO>(ni);
      if (tok >= ntok) continue;
#pragma unroll
      for (int mi = 0; mi < KO::MI; ++mi)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int m = mrow0 + mi * 32 + 8 * g;
          if (m >= mrows) continue;
          const f32x16_t& a = acc[0][mi][ni];
          st4<T>(sg.out, ob + (t0 + tok) * d + m0 + m, a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]);
        }
    }
    return;
  }

  if constexpr (sizeof(T) == 2 && !NARROW && !__is_same(T, _Float16)) {
    if (sg.kind == BWD_GRAD_UPD) {
      grad_update_tile<T>(sg, inst, rr, d, h, smem);
      return;
    }
  }

  const int64_t kb = (int64_t)split * sg.split_len;
  int64_t klen = sg.rows - kb;
  if (klen > sg.split_len) klen = sg.split_len;
  if (klen < 0) klen = 0;
  float* part = reinterpret_cast<float*>(sg.out) + split * sg.out_split + inst * sg.out_inst;
  const int64_t dh = (int64_t)d * h;
  if (sg.kind == BWD_GRAD13) {
    // P1[j, m] = sum_i (eta dz1)[i, j] K[i, m];  P3 likewise with eta dz3
    const int64_t r0 = (int64_t)(rr / sg.tiles_n) * K13::ROWS_A;
    const int64_t c0 = (int64_t)(rr % sg.tiles_n) * K13::ROWS_B;
    const int64_t mrows = h - r0, ncols = d - c0;
    const View ops[3] = {view_mn(sg.a0, inst, r0, kb, mrows, klen, esz), view_mn(sg.a1, inst, r0, kb, mrows, klen, esz),
                         view_mn(sg.b0, inst, c0, kb, ncols, klen, esz)};
    Acc<K13> acc;
    mainloop<T, K13>(smem, ops, klen, acc);
#pragma unroll
    for (int mi = 0; mi < K13::MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < K13::NI; ++ni) {
        const int j = acc_col<K13>(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row<K13>(mi, r);
          if (i < mrows && j < ncols) {
            const int64_t idx = (r0 + i) * d + c0 + j;
            part[idx] = acc[0][mi][ni][r];
            part[2 * dh + idx] = acc[1][mi][ni][r];
          }
        }
      }
    if (sg.sumsq) {
      const float2 t = tile_sumsq<K13>(acc, smem);
      if (threadIdx.x == 0) {
        sg.sumsq[((int64_t)inst * sg.spi + 0) * sg.sumsq_stride + rr] = t.x;
        sg.sumsq[((int64_t)inst * sg.spi + 2) * sg.sumsq_stride + rr] = t.y;
      }
    }
  } else {
    // P2[m, j] = sum_i V[i, m] (eta hidden)[i, j]
    const int64_t r0 = (int64_t)(rr / sg.tiles_n) * K2::ROWS_A;
    const int64_t c0 = (int64_t)(rr % sg.tiles_n) * K2::ROWS_B;
    const int64_t mrows = d - r0, ncols = h - c0;
    const View ops[2] = {view_mn(sg.a0, inst, r0, kb, mrows, klen, esz), view_mn(sg.b0, inst, c0, kb, ncols, klen, esz)};
    Acc<K2> acc;
    mainloop<T, K2>(smem, ops, klen, acc);
#pragma unroll
    for (int mi = 0; mi < K2::MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < K2::NI; ++ni) {
        const int j = acc_col<K2>(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row<K2>(mi, r);
          if (i < mrows && j < ncols) part[sg.out_off + (r0 + i) * h + c0 + j] = acc[0][mi][ni][r];
        }
      }
    if (sg.sumsq) {
      const float2 t = tile_sumsq<K2>(acc, smem);
      if (threadIdx.x == 0) sg.sumsq[((int64_t)inst * sg.spi + sg.sumsq_j) * sg.sumsq_stride + rr] = t.x;
    }
  }
}

template <typename T, bool NARROW>
__global__ __launch_bounds__(Kinds<T>::Out::THREADS) void k_bwd(const BwdArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[bwd_smem<T, NARROW>()];
  bwd_body<T, NARROW>(args, blockIdx.x, smem);
}

// ===========================================================================
// Weight update

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// One wave per row of W1 (length d), W2 (length h) or W3 (length d):
//   U = W + sum_split P  (P = -g, the negated gradient or its Newton-Schulz image)
//   W <- U * ||W_row|| / ||U_row||       (§3.2 weight normalisation; Alg. 1)
// With momentum (App. A, momentum for test-time optimizers; Table 3) the sum
// first goes through the state: Y = sum P - bbar M = -(bbar M + g), M <- -Y,
// U = W + Y.
// Lane l owns the float4 vectors l, l+64, ... of the row (NV per lane at most);
// every load is issued unconditionally (clamped index, zeroed after) so a row
// costs one round trip to memory, not one per vector.
template <typename T, int NV>
__global__ __launch_bounds__(256) void k_update(const UpdArgs a) {
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wave >= a.rows_total) return;
  const int rows_inst = a.nmat == 1 ? a.h : 2 * a.h + a.d;
  const int inst = wave / rows_inst;
  int r = wave - inst * rows_inst;
  int mat, L;
  if (r < a.h) {
    mat = 0; L = a.d;
  } else if (r < a.h + a.d) {
    mat = 1; r -= a.h; L = a.h;
  } else {
    mat = 2; r -= a.h + a.d; L = a.d;
  }
  const int nv = L >> 2;
  const int64_t dh = (int64_t)a.d * a.h;
  const int64_t off = inst * dh + (int64_t)r * L;
  float4* W = reinterpret_cast<float4*>(a.W[mat] + off);
  const float4* Wi = reinterpret_cast<const float4*>((a.Wsrc[mat] ? a.Wsrc[mat] : a.W[mat]) + off);
  const float4* P = reinterpret_cast<const float4*>(a.step + inst * a.nmat * dh + mat * dh + (int64_t)r * L);
  const int64_t ps = a.step_split >> 2;
  float4* Mv = a.M[0] ? reinterpret_cast<float4*>(a.M[mat] + off) : nullptr;
  float4 w[NV], u[NV], m[NV];
#pragma unroll
  for (int t = 0; t < NV; ++t) {
    const int i = lane + 64 * t;
    w[t] = Wi[i < nv ? i : 0];
    u[t] = P[i < nv ? i : 0];
    if (Mv) m[t] = Mv[i < nv ? i : 0];
  }
  for (int s = 1; s < a.nsplit; ++s) {
#pragma unroll
    for (int t = 0; t < NV; ++t) {
      const int i = lane + 64 * t;
      const float4 q = P[s * ps + (i < nv ? i : 0)];
      u[t].x += q.x; u[t].y += q.y; u[t].z += q.z; u[t].w += q.w;
    }
  }
  if (Mv) {
    const float bb = a.bbar[(int64_t)inst * a.bbar_stride];
#pragma unroll
    for (int t = 0; t < NV; ++t) {
      const int i = lane + 64 * t;
      u[t].x = fmaf(-bb, m[t].x, u[t].x);
      u[t].y = fmaf(-bb, m[t].y, u[t].y);
      u[t].z = fmaf(-bb, m[t].z, u[t].z);
      u[t].w = fmaf(-bb, m[t].w, u[t].w);
      if (i < nv) Mv[i] = make_float4(-u[t].x, -u[t].y, -u[t].z, -u[t].w);
    }
  }
  float sw = 0.f, su = 0.f;
#pragma unroll
  for (int t = 0; t < NV; ++t) {
    if (lane + 64 * t >= nv) {
      w[t] = make_float4(0.f, 0.f, 0.f, 0.f);
      u[t] = w[t];
    }
    u[t].x += w[t].x; u[t].y += w[t].y; u[t].z += w[t].z; u[t].w += w[t].w;
    sw += w[t].x * w[t].x + w[t].y * w[t].y + w[t].z * w[t].z + w[t].w * w[t].w;
    su += u[t].x * u[t].x + u[t].y * u[t].y + u[t].z * u[t].z + u[t].w * u[t].w;
  }
  sw = wave_sum(sw);
  su = wave_sum(su);
  const float scale = sqrtf(sw) / sqrtf(su);
#pragma unroll
  for (int t = 0; t < NV; ++t) {
    const int i = lane + 64 * t;
    if (i < nv) {
      const float4 x = make_float4(u[t].x * scale, u[t].y * scale, u[t].z * scale, u[t].w * scale);
      W[i] = x;
      if constexpr (sizeof(T) == 2) {
        typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4_t;
        const bf16x4_t b = {(__bf16)x.x, (__bf16)x.y, (__bf16)x.z, (__bf16)x.w};
        reinterpret_cast<bf16x4_t*>(reinterpret_cast<__bf16*>(a.Wb[mat]) + off)[i] = b;
      }
    }
  }
}

// n4 16-byte vectors of every matrix (d*h is a multiple of 64).
__global__ __launch_bounds__(256) void k_prep(const float* w1, const float* w2, const float* w3, __bf16* b1,
                                              __bf16* b2, __bf16* b3, int64_t n4) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n4) {
    const float4 a = reinterpret_cast<const float4*>(w1)[i];
    st4<__bf16>(b1, 4 * i, a.x, a.y, a.z, a.w);
    if (w2) {   // null for a single fast-weight matrix
      const float4 b = reinterpret_cast<const float4*>(w2)[i], c = reinterpret_cast<const float4*>(w3)[i];
      st4<__bf16>(b2, 4 * i, b.x, b.y, b.z, b.w);
      st4<__bf16>(b3, 4 * i, c.x, c.y, c.z, c.w);
    }
  }
}

// eta_i * k_i for tokens [0, n) of every instance (the linear fast weight's
// gradient operand), rows of d elements, 16 bytes per lane: out [BH][C][d].
// IX: index type of the divisions (32 bits when every index fits; a 64-bit
// division per 16-byte vector costs more than the vector's traffic).
template <typename T, typename IX>
__global__ __launch_bounds__(256) void k_scale_rows(const T* k, const float* eta, T* out, int64_t n, int d,
                                                    int64_t k_inst, int64_t eta_inst, int64_t out_inst, int64_t total) {
  constexpr int EPV = 16 / sizeof(T);
  const IX vpr = (IX)(d / EPV);   // 16-byte vectors per row
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const IX ii = (IX)i, rowi = ii / vpr, insti = rowi / (IX)n;
    const int64_t row = rowi, inst = insti, t = (int64_t)(rowi - insti * (IX)n);
    const int c = (int)(ii - rowi * vpr) * EPV;
    const float e = eta[inst * eta_inst + t];
    typedef __attribute__((ext_vector_type(EPV))) T tv;
    const tv x = *reinterpret_cast<const tv*>(k + inst * k_inst + t * d + c);
    tv y;
#pragma unroll
    for (int j = 0; j < EPV; ++j) y[j] = (T)(e * (float)x[j]);
    *reinterpret_cast<tv*>(out + inst * out_inst + t * d + c) = y;
  }
}

// ===========================================================================
// Newton-Schulz (Muon)

// One Newton-Schulz product over every matrix of the chunk (see NsKind).
// Newton-Schulz products. Every product is computed as the transpose of
// what is stored: element (r, c) of the tile-space product goes to row c,
// column r of the destination, so that the four consecutive accumulator rows
// a lane holds become four consecutive elements of one stored row (one 16-byte
// fp32 / 8-byte 16-bit access). The Gram and polynomial products are
// symmetric, so their transposes are themselves; the update product runs with
// swapped operands (tile rows = Y columns, tile columns = Y rows).
// Newton-Schulz epilogue (16-bit operand copies): the fp32 tile goes through
// LDS in two halves (the wave columns of ni = 0, then ni = 1), WN * 32 stored
// rows of ROWS_A floats each, so that every lane then moves 16 contiguous
// bytes and a wave covers whole 1 KiB row segments: of A32 / Y32 (read and
// written as fp32) and of the fp16 copies. Written straight from the MFMA
// layout, each store instruction touched 32 rows 32 bytes at a time, and the
// epilogue took longer than the product. 16-byte chunks are XOR-swizzled by
// the staged row so that the column-wise writes and the row-wise reads are
// both free of bank conflicts. With `mirror` (an off-diagonal tile of a
// symmetric product computed for the upper triangle only) the Gram and
// polynomial tiles are also written untransposed, to rows i0 + r and columns
// j0 + c: each lane gathers four consecutive staged rows of one tile row
// (compiled in with MIRROR only: the 128 x 128 kinds).
template <typename T, class KK, bool MIRROR>
__device__ __forceinline__ void ns_epilogue_staged(const Acc<KK>& acc, uint8_t* smem, const NsArgs& args, int kind,
                                                   int64_t ld, int64_t i0, int64_t j0, int64_t mrows, int64_t ncols,
                                                   void* Abw, void* A2w, float* Y32, void* Yout, void* Bbw,
                                                   bool mirror) {
  constexpr int R = KK::ROWS_A;                  // tile rows = stored columns
  constexpr int SR = KK::WN * 32;                // staged stored rows per half
  constexpr int CPR = R / 4;                     // 16-byte chunks per staged row
  constexpr int PER = SR * CPR / KK::THREADS;    // chunks per thread per half
  static_assert(KK::NI == 2 && SR * R * 4 <= KK::NSTAGE * KK::STAGE && (SR * CPR) % KK::THREADS == 0 &&
                    (CPR & (CPR - 1)) == 0, "staging shape");
  float* st = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63;
  const bool gram = kind == NS_GRAM_K || kind == NS_GRAM_MN;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    // stage: lane holds rows r..r+3 (stored columns) of tile column c (stored row)
    const int sr = wave_n<KK>() * 32 + (lane & 31);
#pragma unroll
    for (int mi = 0; mi < KK::MI; ++mi)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int r = acc_row<KK>(mi, 4 * g);
        const f32x16_t& a = acc[0][mi][half];
        *reinterpret_cast<float4*>(st + sr * R + (((r >> 2) ^ (sr & (CPR - 1))) << 2)) =
            make_float4(a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]);
      }
    lds_barrier();
    int64_t gidx[PER];
    bool ok[PER];
    int dgn[PER];
    float4 old[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = i * KK::THREADS + threadIdx.x;
      const int srow = q / CPR, ch = q % CPR;
      const int c = (srow / 32) * (KK::NI * 32) + half * 32 + (srow & 31);   // stored row in the tile
      ok[i] = c < ncols && ch * 4 < mrows;
      gidx[i] = (j0 + c) * ld + i0 + ch * 4;
      dgn[i] = (int)(j0 + c - (i0 + ch * 4));
      if (ok[i] && !gram && kind != NS_POLY) old[i] = *reinterpret_cast<const float4*>(Y32 + gidx[i]);
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = i * KK::THREADS + threadIdx.x;
      const int srow = q / CPR, ch = q % CPR;
      const float4 v = *reinterpret_cast<const float4*>(st + srow * R + ((ch ^ (srow & (CPR - 1))) << 2));
      if (!ok[i]) continue;
      if (gram) {
        st4<T>(Abw, gidx[i], v.x, v.y, v.z, v.w);
        // c A + b I, the polynomial's second factor: element e of the four is
        // on the diagonal when the stored row minus the first column is e
        const int dg = dgn[i];
        st4<T>(A2w, gidx[i], args.cc * v.x + (dg == 0 ? args.cb : 0.0f), args.cc * v.y + (dg == 1 ? args.cb : 0.0f),
               args.cc * v.z + (dg == 2 ? args.cb : 0.0f), args.cc * v.w + (dg == 3 ? args.cb : 0.0f));
      } else if (kind == NS_POLY) {
        st4<T>(Bbw, gidx[i], v.x, v.y, v.z, v.w);
      } else {
        const float4 o = old[i];
        const float4 y = make_float4(args.ca * o.x + v.x, args.ca * o.y + v.y, args.ca * o.z + v.z,
                                     args.ca * o.w + v.w);
        *reinterpret_cast<float4*>(Y32 + gidx[i]) = y;
        if (Yout) st4<T>(Yout, gidx[i], y.x, y.y, y.z, y.w);   // none after the last step
      }
    }
    if (MIRROR && mirror) {
      // staged rows 4 s4 .. 4 s4 + 3 are tile columns c0 .. c0 + 3 (one 32-block)
      constexpr int S4 = SR / 4;
      constexpr int PERM = R * S4 / KK::THREADS;
      static_assert((R * S4) % KK::THREADS == 0, "mirror shape");
#pragma unroll
      for (int i = 0; i < PERM; ++i) {
        const int q = i * KK::THREADS + threadIdx.x;
        const int r = q / S4, s0 = 4 * (q % S4);
        const int c0 = (s0 / 32) * (KK::NI * 32) + half * 32 + (s0 & 31);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int sr = s0 + e;
          v[e] = st[sr * R + ((((r >> 2) ^ (sr & (CPR - 1)))) << 2) + (r & 3)];
        }
        if (r >= mrows || c0 >= ncols) continue;
        const int64_t g = (i0 + r) * ld + j0 + c0;
        if (gram) {
          st4<T>(Abw, g, v[0], v[1], v[2], v[3]);
          st4<T>(A2w, g, args.cc * v[0], args.cc * v[1], args.cc * v[2], args.cc * v[3]);   // off the diagonal
        } else {
          st4<T>(Bbw, g, v[0], v[1], v[2], v[3]);
        }
      }
    }
    if (half == 0) lds_barrier();   // every wave has read the first half
  }
}

// The last Newton-Schulz step of square matrices fused with the weight
// update (Muon, §3.2; App. A): 128 whole rows of X5 = a X4 + B X4 per
// workgroup (B X4 from the fp16 copies, a X4 from the fp32 iterate), then the
// normalised update of the same rows of W with X5 as the step (update_rows):
// X5 never goes to memory and no separate update launch runs.
__global__ __launch_bounds__(KNsRow16::THREADS) void k_ns_final(const NsFinalArgs args) {
  using KR = KNsRow16;
  __shared__ __attribute__((aligned(16))) uint8_t smem[smem_bytes<_Float16, KR>()];
  const int tiles = (args.m + KR::ROWS_A - 1) / KR::ROWS_A;
  const int bid = xcd_remap(blockIdx.x, args.nblocks);
  const int slot = bid / tiles, tile = bid - slot * tiles;
  const int inst = slot / args.spi, j = slot - inst * args.spi;
  const int64_t r0 = (int64_t)tile * KR::ROWS_A;
  const int64_t mrows = args.m - r0;
  const Operand b = {reinterpret_cast<const uint8_t*>(args.Bb) + (int64_t)slot * args.astride * 2, args.m, 0};
  const Operand x = {reinterpret_cast<const uint8_t*>(args.Yin) + (int64_t)slot * args.ystride * 2, args.m, 0};
  const View ops[2] = {view_k(b, 0, r0, 0, mrows, args.m, 2), view_mn(x, 0, 0, 0, args.m, args.m, 2)};
  Acc<KR> acc;
  mainloop<_Float16, KR>(smem, ops, args.m, acc);
  const int64_t off = (int64_t)inst * args.ystride + r0 * args.m;
  update_rows<KR, false, true>(acc, args.W[j] + off, reinterpret_cast<__bf16*>(args.Wb[j]) + off, nullptr, 0.f, mrows,
                               args.m, smem, args.Y32 + (int64_t)slot * args.ystride + r0 * args.m, args.ca);
}

template <typename T, bool BIG>
__global__ __launch_bounds__((NsKinds<T, BIG>::K::THREADS)) void k_ns(const NsArgs args) {
  using KK = typename NsKinds<T, BIG>::K;
  using KM = typename NsKinds<T, BIG>::MN;
  using KT = typename NsKinds<T, BIG>::TY;
  static_assert(KK::THREADS == KM::THREADS && KK::THREADS == KT::THREADS && KK::ROWS_A == KM::ROWS_A &&
                    KK::ROWS_A == KT::ROWS_A && KK::ROWS_B == KT::ROWS_B && KK::MI == KT::MI && KK::NI == KM::NI,
                "one tile and accumulator shape per launch");
  __shared__ __attribute__((aligned(16)))
  uint8_t smem[cmax(smem_bytes<T, KK>(), cmax(smem_bytes<T, KM>(), smem_bytes<T, KT>()))];
  constexpr int esz = sizeof(T);
  int bid = blockIdx.x;
  const bool first = bid < args.seg[0].nblocks;
  const NsSeg& sg = first ? args.seg[0] : args.seg[1];
  if (!first) bid -= args.seg[0].nblocks;
  bid = xcd_remap(bid, sg.nblocks);
  const int per = sg.tri ? sg.tiles_m * (sg.tiles_m + 1) / 2 : sg.tiles_m * sg.tiles_n;
  const int q = bid / per;
  const int rr = bid - q * per;
  int ti = rr / sg.tiles_n, tj = rr % sg.tiles_n;
  if (sg.tri) {   // row ti of the upper triangle holds tiles_m - ti tiles
    ti = 0;
    int left = rr;
    while (left >= sg.tiles_m - ti) {
      left -= sg.tiles_m - ti;
      ++ti;
    }
    tj = ti + left;
  }
  const int64_t i0 = (int64_t)ti * KK::ROWS_A, j0 = (int64_t)tj * KK::ROWS_B;
  const int64_t slot = (int64_t)(q / sg.group) * args.spi + sg.slot_off[q % sg.group];
  const int m = args.m, ldy = sg.ldy;
  const int64_t mrows = sg.M - i0, ncols = sg.N - j0;
  float* Y32 = args.Y32 + slot * args.ystride;
  const uint8_t* Yin = reinterpret_cast<const uint8_t*>(args.Yin) + slot * args.ystride * esz;
  void* Yout = args.Yout ? reinterpret_cast<uint8_t*>(args.Yout) + slot * args.ystride * esz : nullptr;
  const uint8_t* Ab = reinterpret_cast<const uint8_t*>(args.Ab) + slot * args.astride * esz;
  void* Abw = reinterpret_cast<uint8_t*>(args.Ab) + slot * args.astride * esz;
  const uint8_t* A2 = reinterpret_cast<const uint8_t*>(args.A2b) + slot * args.astride * esz;
  void* A2w = reinterpret_cast<uint8_t*>(args.A2b) + slot * args.astride * esz;
  const uint8_t* Bb = reinterpret_cast<const uint8_t*>(args.Bb) + slot * args.astride * esz;
  void* Bbw = reinterpret_cast<uint8_t*>(args.Bb) + slot * args.astride * esz;
  Acc<KK> acc;   // same accumulator shape for every NS kind
  const int kind = sg.kind;
  if (kind == NS_GRAM_K) {          // A = Y Y^T (Y wide)
    const View ops[2] = {View{Yin + i0 * ldy * esz, (int64_t)ldy * esz, mrows, sg.K},
                         View{Yin + j0 * ldy * esz, (int64_t)ldy * esz, ncols, sg.K}};
    mainloop<T, KK>(smem, ops, sg.K, acc);
  } else if (kind == NS_GRAM_MN) {  // A = Y^T Y (Y tall)
    const View ops[2] = {View{Yin + i0 * esz, (int64_t)ldy * esz, mrows, sg.K},
                         View{Yin + j0 * esz, (int64_t)ldy * esz, ncols, sg.K}};
    mainloop<T, KM>(smem, ops, sg.K, acc);
  } else if (kind == NS_POLY) {     // A (c A + b I) = b A + c A A (both symmetric: A A2^T)
    const View ops[2] = {View{Ab + i0 * m * esz, (int64_t)m * esz, mrows, sg.K},
                         View{A2 + j0 * m * esz, (int64_t)m * esz, ncols, sg.K}};
    mainloop<T, KK>(smem, ops, sg.K, acc);
  } else if (kind == NS_UPD_BY) {   // (B Y)^T = Y^T B (Y wide, B symmetric): rows = Y columns
    const View ops[2] = {View{Yin + i0 * esz, (int64_t)ldy * esz, mrows, sg.K},
                         View{Bb + j0 * m * esz, (int64_t)m * esz, ncols, sg.K}};
    mainloop<T, KT>(smem, ops, sg.K, acc);
  } else {                          // (Y B)^T = B Y^T (Y tall): rows = Y columns
    const View ops[2] = {View{Bb + i0 * m * esz, (int64_t)m * esz, mrows, sg.K},
                         View{Yin + j0 * ldy * esz, (int64_t)ldy * esz, ncols, sg.K}};
    mainloop<T, KK>(smem, ops, sg.K, acc);
  }
  const bool gram = kind == NS_GRAM_K || kind == NS_GRAM_MN;
  const int64_t ld = (gram || kind == NS_POLY) ? m : ldy;
  if constexpr (sizeof(T) == 2) {
    ns_epilogue_staged<T, KK, !BIG>(acc, smem, args, kind, ld, i0, j0, mrows, ncols, Abw, A2w, Y32, Yout, Bbw,
                                    sg.tri && ti != tj && (gram || kind == NS_POLY));
    return;
  }
#pragma unroll
  for (int mi = 0; mi < KK::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < KK::NI; ++ni) {
      const int c = acc_col<KK>(ni);
      if (c >= ncols) continue;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int r = acc_row<KK>(mi, 4 * g);    // rows r .. r+3 of the tile
        if (r >= mrows) continue;
        const f32x16_t& a = acc[0][mi][ni];
        const float v0 = a[4 * g], v1 = a[4 * g + 1], v2 = a[4 * g + 2], v3 = a[4 * g + 3];
        const int64_t idx = (j0 + c) * ld + i0 + r;   // stored row j0+c, columns i0+r ..
        if (gram) {
          st4<T>(Abw, idx, v0, v1, v2, v3);
          const int dg = (int)(j0 + c - (i0 + r));   // c A + b I (see ns_epilogue_staged)
          st4<T>(A2w, idx, args.cc * v0 + (dg == 0 ? args.cb : 0.0f), args.cc * v1 + (dg == 1 ? args.cb : 0.0f),
                 args.cc * v2 + (dg == 2 ? args.cb : 0.0f), args.cc * v3 + (dg == 3 ? args.cb : 0.0f));
        } else if (kind == NS_POLY) {
          st4<T>(Bbw, idx, v0, v1, v2, v3);
        } else {
          const float4 o = *reinterpret_cast<const float4*>(Y32 + idx);
          const float4 y =
              make_float4(args.ca * o.x + v0, args.ca * o.y + v1, args.ca * o.z + v2, args.ca * o.w + v3);
          *reinterpret_cast<float4*>(Y32 + idx) = y;
          if (Yout) st4<T>(Yout, idx, y.x, y.y, y.z, y.w);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// Whole Newton-Schulz iteration of one small matrix per workgroup (Gram size
// m <= 128, long side n <= 256), from the summed gradient to the updated
// weights: X0 = G / (||G||_F + eps) is formed in registers, the fp16 iterate
// X, Gram A and polynomial B stay in LDS (64 + 32 + 32 KiB), the fp32 iterate
// in registers, and the weight update takes the result as its step. Per step:
//   A = X X^T   (kept in fp32 registers, fp16 copy to LDS)
//   B = b A + c A A
//   X <- a X + B X
// X is held in its stored orientation Y [SR x SC] (wide: Y = X, tall: Y =
// X^T), zero-padded to 128 x 256 (or 256 x 128). Every product is computed in
// the orientation whose lanes own four consecutive elements of a stored row:
// A and B are symmetric, and the last product's tile rows are Y's columns.
// LDS rows are XOR-swizzled by fsw(row) on their 16-byte chunks, which keeps
// both the K-contiguous fragment reads (16 consecutive rows, one chunk) and
// the transposed reads (4 consecutive rows, two adjacent chunks) conflict-free.
__device__ __forceinline__ int fsw(int row) { return ((row & 7) << 1) | ((row >> 3) & 1); }
__device__ __forceinline__ uint32_t fs_off(int row, int chunk, int pitch) {
  return (uint32_t)(row * pitch + ((chunk ^ fsw(row)) << 4));
}
// K-contiguous fragment: row `row`, 8 K from chunk `chunk`.
__device__ __forceinline__ u32x4_t fs_frag_k(uint32_t base, int row, int chunk, int pitch) {
  return lds_read_b128(base + fs_off(row, chunk, pitch));
}
// Transposed fragment (8 consecutive K of column rb + lane%32 of a tile whose
// K runs down the rows, substep s).
__device__ __forceinline__ u32x4_t fs_frag_tr(uint32_t base, int rb, int s, int pitch) {
  const int lane = threadIdx.x & 63, g = lane >> 4, sl = lane & 15;
  const int mn = rb + 16 * (g & 1) + 4 * (sl & 3);
  const int c = mn >> 3, hb = (mn >> 2) & 1;
  u32x2_t lo, hi;
  {
    const int kr = 16 * s + 8 * (g >> 1) + (sl >> 2);
    const uint32_t a = base + kr * pitch + ((c ^ fsw(kr)) << 4) + (hb << 3);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a));
  }
  {
    const int kr = 16 * s + 8 * (g >> 1) + 4 + (sl >> 2);
    const uint32_t a = base + kr * pitch + ((c ^ fsw(kr)) << 4) + (hb << 3);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(hi) : "v"(a));
  }
  return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
}
// Wait for every LDS read of this wave and make the fragments depend on the
// wait, so that no MFMA reading them can be scheduled above it.
template <int NA, int NB>
__device__ __forceinline__ void lds_ready(u32x4_t (&fa)[NA], u32x4_t (&fb)[NB]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < NA; ++i) asm volatile("" : "+v"(fa[i]));
#pragma unroll
  for (int i = 0; i < NB; ++i) asm volatile("" : "+v"(fb[i]));
}
__device__ __forceinline__ f32x16_t mfma16(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c, 0,
                                                0, 0);
}
// four fp16 values at (row, cols col .. col+3) of a swizzled LDS matrix
__device__ __forceinline__ void fs_put4(uint8_t* base, int row, int col, int pitch, float a, float b, float c, float d) {
  typedef __attribute__((ext_vector_type(4))) _Float16 h4;
  *reinterpret_cast<h4*>(base + fs_off(row, col >> 3, pitch) + (((col >> 2) & 1) << 3)) =
      h4{(_Float16)a, (_Float16)b, (_Float16)c, (_Float16)d};
}

// LDS of one fused Newton-Schulz workgroup: X (padded to 128 x 256 or
// 256 x 128, fp16), A and B (128 x 128 fp16 each); the same for both
// orientations.
constexpr int kNsFusedX = kNsFusedM * kNsFusedN * 2, kNsFusedA = kNsFusedM * kNsFusedM * 2;

template <bool TALL>
__device__ __forceinline__ void ns_fused_body(const NsFusedArgs& a, int q, uint8_t* xs, uint8_t* as_, uint8_t* bs) {
  constexpr int M = kNsFusedM, N = kNsFusedN;
  constexpr int SR = TALL ? N : M, SC = TALL ? M : N;   // padded stored orientation
  constexpr int PX = SC * 2, PA = M * 2;                // LDS pitches (bytes)
  static_assert(SR * PX == kNsFusedX && M * PA == kNsFusedA, "LDS buffers");
  const uint32_t xb = lds_addr(xs), ab = lds_addr(as_), bb = lds_addr(bs);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, half = lane >> 5;
  const int64_t slot = (int64_t)(q / a.group) * a.spi + a.slot_off[q % a.group];
  const int sr = a.rows, sc = a.cols;                   // valid stored rows, columns

  // LDS copy of X zero padded (written below)
  for (int i = tid; i < SR * PX / 16; i += 512) *reinterpret_cast<u32x4_t*>(xs + i * 16) = u32x4_t{0u, 0u, 0u, 0u};
  __syncthreads();
  // The summed gradient into registers, in the tile layout of the update
  // product: tile rows = stored columns (TR rows), tile columns = stored rows (TC)
  constexpr int WM3 = TALL ? 2 : 4, WN3 = TALL ? 4 : 2;   // waves: 64 x 64 each
  const int r3 = (w / WN3) * 64, c3 = (w % WN3) * 64;
  const float* xin = a.src + slot * a.ystride;
  const int nin = a.nsplit;
  f32x16_t x32[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int c = c3 + ni * 32 + (lane & 31);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int r = r3 + mi * 32 + 8 * g + 4 * half;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (c < sr && r < sc)
          for (int sp = 0; sp < nin; ++sp) {
            const float4 p = *reinterpret_cast<const float4*>(xin + sp * a.part_split + (int64_t)c * sc + r);
            v = make_float4(v.x + p.x, v.y + p.y, v.z + p.z, v.w + p.w);
          }
        x32[mi][ni][4 * g] = v.x;
        x32[mi][ni][4 * g + 1] = v.y;
        x32[mi][ni][4 * g + 2] = v.z;
        x32[mi][ni][4 * g + 3] = v.w;
      }
    }
  {
    // X0 = G / (||G||_F + eps): the whole matrix is in this workgroup's
    // registers (padding is zero); the partial sums go through the start of
    // the Gram buffer, which the first step overwrites only after a barrier
    float ss = 0.f;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int e = 0; e < 16; ++e) ss = fmaf(x32[mi][ni][e], x32[mi][ni][e], ss);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    float* red = reinterpret_cast<float*>(as_);
    if (lane == 0) red[w] = ss;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) t += red[i];
    const float inv = 1.0f / (sqrtf(t) + a.eps);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int c = c3 + ni * 32 + (lane & 31);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = r3 + mi * 32 + 8 * g + 4 * half;
#pragma unroll
          for (int e = 0; e < 4; ++e) x32[mi][ni][4 * g + e] *= inv;
          fs_put4(xs, c, r, PX, x32[mi][ni][4 * g], x32[mi][ni][4 * g + 1], x32[mi][ni][4 * g + 2],
                  x32[mi][ni][4 * g + 3]);
        }
      }
  }
  __syncthreads();

  // Gram tile layout: waves 2 x 4 of 64 x 32
  const int r1 = (w >> 2) * 64, c1 = (w & 3) * 32;
  for (int step = 0; step < a.steps; ++step) {
    // ---- A = X X^T (K = N) ----
    f32x16_t a32[2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int e = 0; e < 16; ++e) a32[mi][e] = 0.f;
    for (int s = 0; s < N / 16; ++s) {
      u32x4_t fa[2], fb[1];
      if constexpr (!TALL) {
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) fa[mi] = fs_frag_k(xb, r1 + mi * 32 + (lane & 31), 2 * s + half, PX);
        fb[0] = fs_frag_k(xb, c1 + (lane & 31), 2 * s + half, PX);
      } else {
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) fa[mi] = fs_frag_tr(xb, r1 + mi * 32, s, PX);
        fb[0] = fs_frag_tr(xb, c1, s, PX);
      }
      lds_ready(fa, fb);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) a32[mi] = mfma16(fa[mi], fb[0], a32[mi]);
    }
    // A is symmetric: lane's rows i..i+3 at column j go to row j, columns i..i+3
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        fs_put4(as_, c1 + (lane & 31), r1 + mi * 32 + 8 * g + 4 * half, PA, a32[mi][4 * g], a32[mi][4 * g + 1],
                a32[mi][4 * g + 2], a32[mi][4 * g + 3]);
    lds_barrier();
    // ---- B = b A + c A A (K = M) ----
    f32x16_t t[2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int e = 0; e < 16; ++e) t[mi][e] = 0.f;
    for (int s = 0; s < M / 16; ++s) {
      u32x4_t fa[2], fb[1];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) fa[mi] = fs_frag_k(ab, r1 + mi * 32 + (lane & 31), 2 * s + half, PA);
      fb[0] = fs_frag_k(ab, c1 + (lane & 31), 2 * s + half, PA);
      lds_ready(fa, fb);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) t[mi] = mfma16(fa[mi], fb[0], t[mi]);
    }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = a.cb * a32[mi][4 * g + e] + a.cc * t[mi][4 * g + e];
        fs_put4(bs, c1 + (lane & 31), r1 + mi * 32 + 8 * g + 4 * half, PA, v[0], v[1], v[2], v[3]);
      }
    lds_barrier();
    // ---- X <- a X + B X (K = M), tile rows = stored columns ----
    f32x16_t u[2][2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int e = 0; e < 16; ++e) u[mi][ni][e] = 0.f;
    for (int s = 0; s < M / 16; ++s) {
      u32x4_t fa[2], fb[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        if constexpr (!TALL) fa[mi] = fs_frag_tr(xb, r3 + mi * 32, s, PX);   // X[k][j], k down the rows
        else fa[mi] = fs_frag_k(bb, r3 + mi * 32 + (lane & 31), 2 * s + half, PA);   // B[i][k]
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        if constexpr (!TALL) fb[ni] = fs_frag_k(bb, c3 + ni * 32 + (lane & 31), 2 * s + half, PA);   // B[i][k]
        else fb[ni] = fs_frag_k(xb, c3 + ni * 32 + (lane & 31), 2 * s + half, PX);   // Y[j][k] = X[k][j]
      }
      lds_ready(fa, fb);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) u[mi][ni] = mfma16(fa[mi], fb[ni], u[mi][ni]);
    }
    lds_barrier();   // every wave is done reading X before it is overwritten
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int c = c3 + ni * 32 + (lane & 31);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = r3 + mi * 32 + 8 * g + 4 * half;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = a.ca * x32[mi][ni][4 * g + e] + u[mi][ni][4 * g + e];
            x32[mi][ni][4 * g + e] = v[e];
          }
          fs_put4(xs, c, r, PX, v[0], v[1], v[2], v[3]);
        }
      }
    lds_barrier();
  }
  {
    // The weight update of this matrix with X as the step (§3.2 weight
    // normalisation; Muon's update, App. A): a lane holds 32 columns of stored
    // rows c (ni = 0, 1); row sums over the lane, its partner half (lane ^ 32)
    // and the WM3 wave rows (through LDS, free after the last step's barrier)
    const int j = a.slot_off[q % a.group];
    const int64_t woff = (int64_t)(q / a.group) * a.ystride;
    float* Wj = a.W[j] + woff;
    __bf16* Wbj = reinterpret_cast<__bf16*>(a.Wb[j]) + woff;
    float sw[2] = {0.f, 0.f}, su[2] = {0.f, 0.f};
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int c = c3 + ni * 32 + (lane & 31);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = r3 + mi * 32 + 8 * g + 4 * half;
          float4 wv = make_float4(0.f, 0.f, 0.f, 0.f);
          if (c < sr && r < sc) wv = *reinterpret_cast<const float4*>(Wj + (int64_t)c * sc + r);
          const float wa[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float u = wa[e] + x32[mi][ni][4 * g + e];
            x32[mi][ni][4 * g + e] = u;
            sw[ni] = fmaf(wa[e], wa[e], sw[ni]);
            su[ni] = fmaf(u, u, su[ni]);
          }
        }
      sw[ni] += __shfl_xor(sw[ni], 32, 64);
      su[ni] += __shfl_xor(su[ni], 32, 64);
    }
    float* red = reinterpret_cast<float*>(as_);   // [WM3][SR][2]
    const int wr = w / WN3;
    if (half == 0)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int c = c3 + ni * 32 + (lane & 31);
        red[(wr * SR + c) * 2] = sw[ni];
        red[(wr * SR + c) * 2 + 1] = su[ni];
      }
    __syncthreads();
    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4_t;
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int c = c3 + ni * 32 + (lane & 31);
      float tw = 0.f, tu = 0.f;
#pragma unroll
      for (int k = 0; k < WM3; ++k) {
        tw += red[(k * SR + c) * 2];
        tu += red[(k * SR + c) * 2 + 1];
      }
      const float f = sqrtf(tw) / sqrtf(tu);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = r3 + mi * 32 + 8 * g + 4 * half;
          if (c < sr && r < sc) {
            const float4 x = make_float4(x32[mi][ni][4 * g] * f, x32[mi][ni][4 * g + 1] * f,
                                         x32[mi][ni][4 * g + 2] * f, x32[mi][ni][4 * g + 3] * f);
            *reinterpret_cast<float4*>(Wj + (int64_t)c * sc + r) = x;
            *reinterpret_cast<bf16x4_t*>(Wbj + (int64_t)c * sc + r) =
                bf16x4_t{(__bf16)x.x, (__bf16)x.y, (__bf16)x.z, (__bf16)x.w};
          }
        }
    }
  }
}

template <bool TALL>
__global__ __launch_bounds__(512) void k_ns_fused(const NsFusedArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t xs[kNsFusedX];
  __shared__ __attribute__((aligned(16))) uint8_t as_[kNsFusedA];
  __shared__ __attribute__((aligned(16))) uint8_t bs[kNsFusedA];
  ns_fused_body<TALL>(a, blockIdx.x, xs, as_, bs);
}

// Both matrix groups of an instance set in one launch (W1 and W3, then W2, in
// their own orientations): blocks below a0.nblocks take a0, the rest a1, so
// that the matrices of both orientations fill the chip together.
template <bool TALL0, bool TALL1>
__global__ __launch_bounds__(512) void k_ns_fused_pair(const NsFusedArgs a0, const NsFusedArgs a1) {
  __shared__ __attribute__((aligned(16))) uint8_t xs[kNsFusedX];
  __shared__ __attribute__((aligned(16))) uint8_t as_[kNsFusedA];
  __shared__ __attribute__((aligned(16))) uint8_t bs[kNsFusedA];
  const int q = blockIdx.x;
  if (q < a0.nblocks) ns_fused_body<TALL0>(a0, q, xs, as_, bs);
  else ns_fused_body<TALL1>(a1, q - a0.nblocks, xs, as_, bs);
}

// The small-matrix Newton-Schulz of both groups together with the output
// tiles of the same chunk's apply (o = W2 hidden, 16-bit narrow shapes): the
// output reads the pre-update copy of W2 while the Newton-Schulz blocks write
// the updated copies into the other copy set, so the two are independent and
// the output tiles take the CUs that the one-workgroup-per-matrix
// Newton-Schulz leaves idle. Blocks below a0.nblocks + a1.nblocks run the
// Newton-Schulz, the rest the output tiles.
template <bool TALL0, bool TALL1>
__global__ __launch_bounds__(512) void k_ns_fused_pair_out(const NsFusedArgs a0, const NsFusedArgs a1,
                                                           const BwdArgs out) {
  static_assert(KOutN16::THREADS == 512, "one block size");
  constexpr int kNs = kNsFusedX + 2 * kNsFusedA;
  __shared__ __attribute__((aligned(16))) uint8_t smem[cmax(kNs, bwd_smem<__bf16, true>())];
  const int q = blockIdx.x;
  if (q < a0.nblocks) ns_fused_body<TALL0>(a0, q, smem, smem + kNsFusedX, smem + kNsFusedX + kNsFusedA);
  else if (q < a0.nblocks + a1.nblocks)
    ns_fused_body<TALL1>(a1, q - a0.nblocks, smem, smem + kNsFusedX, smem + kNsFusedX + kNsFusedA);
  else bwd_body<__bf16, true>(out, q - a0.nblocks - a1.nblocks, smem);
}

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) t += red[i];
  __syncthreads();
  return t;
}

// Sum the split-K partials of every gradient and the per-block sums of squares.
// With momentum the iterate is Y = sum P - bbar M = -(bbar M + g) and M <- -Y
// (App. A, momentum; Table 3, Muon row): Newton-Schulz then runs on the state.
__global__ __launch_bounds__(256) void k_ns_prep(const NsPrepArgs a) {
  __shared__ float red[4];
  const int slot = blockIdx.x / a.blocks_per_slot;
  const int blk = blockIdx.x - slot * a.blocks_per_slot;
  const int64_t base = (int64_t)slot * a.dh;
  const int inst = slot / a.spi, j = slot - a.spi * (slot / a.spi);
  float* Ms = a.M[0] ? a.M[j] + (int64_t)inst * a.dh : nullptr;
  const float bb = Ms ? a.bbar[(int64_t)inst * a.bbar_stride] : 0.f;
  // 16 bytes per lane (d*h is a multiple of 4, and so is every offset)
  float ss = 0.f;
  for (int e = 4 * threadIdx.x; e < kNsBlockElems; e += 4 * 256) {
    const int64_t idx = (int64_t)blk * kNsBlockElems + e;
    if (idx < a.dh) {
      float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s = 0; s < a.nsplit; ++s) {
        const float4 p = *reinterpret_cast<const float4*>(a.part + s * a.part_split + base + idx);
        g = make_float4(g.x + p.x, g.y + p.y, g.z + p.z, g.w + p.w);
      }
      if (Ms) {
        const float4 m = *reinterpret_cast<const float4*>(Ms + idx);
        g = make_float4(fmaf(-bb, m.x, g.x), fmaf(-bb, m.y, g.y), fmaf(-bb, m.z, g.z), fmaf(-bb, m.w, g.w));
        *reinterpret_cast<float4*>(Ms + idx) = make_float4(-g.x, -g.y, -g.z, -g.w);
      }
      *reinterpret_cast<float4*>(a.Y32 + base + idx) = g;
      ss += g.x * g.x + g.y * g.y + g.z * g.z + g.w * g.w;
    }
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) a.sumsq[(int64_t)slot * a.blocks_per_slot + blk] = ss;
}

// X0 = G / (||G||_F + eps), fp32 iterate and operand copy; G is the summed
// gradient (Y32) or, without split and momentum, the gradient partial itself.
template <typename T>
__global__ __launch_bounds__(256) void k_ns_scale(const NsPrepArgs a, void* yb, float eps) {
  __shared__ float red[4];
  const int slot = blockIdx.x / a.blocks_per_slot;
  const int blk = blockIdx.x - slot * a.blocks_per_slot;
  const int64_t base = (int64_t)slot * a.dh;
  const int nsum = a.src ? a.sum_n[slot % a.spi] : a.blocks_per_slot;
  float t = 0.f;
  for (int b = threadIdx.x; b < nsum; b += 256) t += a.sumsq[(int64_t)slot * a.blocks_per_slot + b];
  t = block_sum(t, red);
  const float inv = 1.0f / (sqrtf(t) + eps);
  const float* src = a.src ? a.src : a.Y32;
  for (int e = 4 * threadIdx.x; e < kNsBlockElems; e += 4 * 256) {
    const int64_t idx = (int64_t)blk * kNsBlockElems + e;
    if (idx < a.dh) {
      const float4 g = *reinterpret_cast<const float4*>(src + base + idx);
      const float4 y = make_float4(g.x * inv, g.y * inv, g.z * inv, g.w * inv);
      *reinterpret_cast<float4*>(a.Y32 + base + idx) = y;
      st4<T>(yb, base + idx, y.x, y.y, y.z, y.w);
    }
  }
}

// Chunk mean of the per-token momentum factor (App. A, momentum): one block
// per (instance, chunk), fp64 accumulation.
__global__ __launch_bounds__(256) void k_beta_mean(const BetaArgs a) {
  __shared__ double red[4];
  const int inst = blockIdx.x / a.nchunks;
  const int c = blockIdx.x - inst * a.nchunks;
  const int64_t t0 = a.t0 + c * a.chunk;
  const int64_t t1 = t0 + a.chunk < a.end ? t0 + a.chunk : a.end;
  const float* b = a.beta + (int64_t)inst * a.n_kv;
  double s = 0.0;
  for (int64_t t = t0 + threadIdx.x; t < t1; t += 256) s += (double)b[t];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double tot = red[0] + red[1] + red[2] + red[3];
    a.bbar[(int64_t)inst * a.stride + c] = (float)(tot / (double)(t1 - t0));
  }
}

// ---------------------------------------------------------------------------
// Reverse of the linear fast weight's chunk loop (§5.4 with the §3.1 loss and
// norm-preserving update): the contractions run on the OUT and GRAD2 kinds;
// these kernels are the row-wise and token-wise steps between them.

// Rows of a matrix per workgroup of k_vjp: the rows' cotangent in the operand
// type is staged in LDS (up to 64 KB) to leave as whole segments of the
// transposed copy.
template <typename T, int NV>
constexpr int vjp_rows() {
  return cmax(4, 65536 / (256 * NV * (int)sizeof(T)) > 32 ? 32 : 65536 / (256 * NV * (int)sizeof(T)));
}

template <int NV>
constexpr int vjp_waves() { return NV <= 4 ? 16 : 4; }   // rows of up to 1024 floats: 16 waves in flight

// acc += the split partials of set s at element 4 i of row offset roff
// (lanes past the row pass i = 0 and drop the result).
__device__ __forceinline__ void add_set(const PartSet& s, int64_t inst, int64_t roff, int i, float4& acc) {
  if (!s.p) return;
  const float4* p = reinterpret_cast<const float4*>(s.p + inst * s.inst + roff);
  const int64_t ss = s.split >> 2;
  const float f = s.sign != 0.0f ? s.sign : 1.0f;
  for (int k = 0; k < s.n; ++k) {
    const float4 q = p[k * ss + i];
    acc.x += f * q.x; acc.y += f * q.y; acc.z += f * q.z; acc.w += f * q.w;
  }
}

// Reverse of W' = (n / u) U, U = W + P (P the negated chunk gradient, as
// split partials), vjp_rows() rows of one instance per workgroup, one wave
// per row at a time. From the cotangent G of W' (in place; the pre sets
// join it first), with a = G . U per row:
//   Uh = (n / u) G - (n a / u^3) U,   G <- Uh + (a / (u n)) W  (+ the post set),
// and Uh (the cotangent of U, i.e. minus that of the gradient) in the
// operand type, row-major into Ub and transposed into UT. A zero row norm
// gives the same non-finite values as the forward's division.
template <typename T, int NV>
__device__ __forceinline__ void vjp_body(const VjpArgs& a, int blk, T* tile) {
  constexpr int RR = vjp_rows<T, NV>();
  constexpr int NW = vjp_waves<NV>();
  constexpr int LD = 256 * NV + 4 / (int)sizeof(T);   // one 4-byte word of padding per staged row
  const int L = a.L;
  const int per = (a.R + RR - 1) / RR;
  const int64_t inst = blk / per;
  const int r0 = (int)(blk - inst * per) * RR;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nv = L >> 2;
  T* Ub = reinterpret_cast<T*>(a.Ub);
  T* UT = reinterpret_cast<T*>(a.UT);
  for (int rr = w; rr < RR; rr += NW) {
    const int r = r0 + rr;
    if (r >= a.R) break;
    const int64_t roff = (int64_t)r * L;
    const float4* w4 = reinterpret_cast<const float4*>(a.W + inst * a.w_inst + roff);
    float4* g4 = reinterpret_cast<float4*>(a.G + inst * a.g_inst + roff);
    float4 wv[NV], u[NV], g[NV], ap[NV];
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int t = 0; t < NV; ++t) {
      const int i = lane + 64 * t, ic = i < nv ? i : 0;   // lanes past the row load element 0, then drop it
      wv[t] = w4[ic];
      g[t] = g4[ic];
      u[t] = wv[t];
      ap[t] = z;
      add_set(a.P, inst, roff, ic, u[t]);
      add_set(a.pre[0], inst, roff, ic, g[t]);
      add_set(a.pre[1], inst, roff, ic, g[t]);
      add_set(a.post, inst, roff, ic, ap[t]);
      if (i >= nv) wv[t] = u[t] = g[t] = z;
    }
    float sw = 0.f, su = 0.f, sa = 0.f;
#pragma unroll
    for (int t = 0; t < NV; ++t) {
      sw += wv[t].x * wv[t].x + wv[t].y * wv[t].y + wv[t].z * wv[t].z + wv[t].w * wv[t].w;
      su += u[t].x * u[t].x + u[t].y * u[t].y + u[t].z * u[t].z + u[t].w * u[t].w;
      sa += g[t].x * u[t].x + g[t].y * u[t].y + g[t].z * u[t].z + g[t].w * u[t].w;
    }
    sw = wave_sum(sw);
    su = wave_sum(su);
    sa = wave_sum(sa);
    const float n = sqrtf(sw), uu = sqrtf(su);
    const float c1 = n / uu, c2 = n * sa / (uu * uu * uu), c3 = sa / (uu * n);
#pragma unroll
    for (int t = 0; t < NV; ++t) {
      const int i = lane + 64 * t;
      if (i >= nv) continue;
      const float4 uh = make_float4(c1 * g[t].x - c2 * u[t].x, c1 * g[t].y - c2 * u[t].y,
                                    c1 * g[t].z - c2 * u[t].z, c1 * g[t].w - c2 * u[t].w);
      g4[i] = make_float4(uh.x + c3 * wv[t].x + ap[t].x, uh.y + c3 * wv[t].y + ap[t].y,
                          uh.z + c3 * wv[t].z + ap[t].z, uh.w + c3 * wv[t].w + ap[t].w);
      if (Ub) st4<T>(Ub, inst * a.ub_inst + (int64_t)r * a.ub_ld + 4 * i, uh.x, uh.y, uh.z, uh.w);
      if (a.U32) reinterpret_cast<float4*>(a.U32 + inst * a.u32_inst + roff)[i] = uh;
      T* row = tile + rr * LD + 4 * i;
      row[0] = (T)uh.x;
      row[1] = (T)uh.y;
      row[2] = (T)uh.z;
      row[3] = (T)uh.w;
    }
  }
  if (!UT) return;   // uniform over the launch
  __syncthreads();
  // UT[c][r0 .. r0 + RR): four consecutive rows of the block per store
  constexpr int Q = RR / 4;
  const int rows = a.R - r0 < RR ? a.R - r0 : RR;
  for (int pi = threadIdx.x; pi < L * Q; pi += 64 * NW) {
    const int c = pi / Q, j = 4 * (pi - (pi / Q) * Q);
    if (j >= rows) continue;
    const int64_t o = inst * a.ut_inst + (int64_t)c * a.ut_ld + r0 + j;
    if (j + 4 <= rows && ((o & 3) == 0)) {
      st4<T>(UT, o, (float)tile[j * LD + c], (float)tile[(j + 1) * LD + c], (float)tile[(j + 2) * LD + c],
             (float)tile[(j + 3) * LD + c]);
    } else {
      for (int q = 0; q < 4 && j + q < rows; ++q) UT[o + q] = tile[(j + q) * LD + c];
    }
  }
}

// Up to three matrices' reverses, blocks n0 of the first, n1 of the second,
// then the third's.
template <typename T, int NV>
__global__ __launch_bounds__(64 * vjp_waves<NV>()) void k_vjp(const VjpArgs a0, const VjpArgs a1, const VjpArgs a2,
                                                              int n0, int n1) {
  __shared__ __attribute__((aligned(16))) T tile[vjp_rows<T, NV>() * (256 * NV + 4 / (int)sizeof(T))];
  const int b = blockIdx.x;
  if (b < n0) vjp_body<T, NV>(a0, b, tile);
  else if (b < n0 + n1) vjp_body<T, NV>(a1, b - n0, tile);
  else vjp_body<T, NV>(a2, b - n0 - n1, tile);
}

// Operand copies of fp32 [R x L] matrices, row-major and/or transposed: one
// 64 x 64 tile per block (segments in order, then instances, then tiles),
// read once as float4 rows into LDS and written as runs of four elements
// along the rows of each copy.
struct CopyArgs {
  CopySeg seg[kMaxCopies];
  int first[kMaxCopies + 1];   // first block of each segment
  int n;
};

template <typename T>
__global__ __launch_bounds__(256) void k_copies(const CopyArgs a) {
  __shared__ float tile[64][65];
  int si = 0;
  while (si + 1 < a.n && (int)blockIdx.x >= a.first[si + 1]) ++si;
  const CopySeg& g = a.seg[si];
  const int tr = (g.R + 63) / 64, tl = (g.L + 63) / 64;
  const int64_t b = blockIdx.x - a.first[si];
  const int64_t per = (int64_t)tr * tl;
  const int64_t inst = b / per;
  const int rest = (int)(b - inst * per);
  const int r0 = (rest / tl) * 64, c0 = (rest % tl) * 64;
  const float* src = g.W + inst * g.w_inst;
  const int t = threadIdx.x, q = (t & 15) * 4;
  const int nsum = g.nsum > 1 ? g.nsum : 1;
  const float sign = g.sign != 0.0f ? g.sign : 1.0f;
  for (int k = t >> 4; k < 64; k += 16) {   // row k of the tile, columns q .. q + 3
    const int r = r0 + k, c = c0 + q;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sp = 0; sp < nsum; ++sp) {
      const float* sr = src + sp * g.split;
      float e[4] = {0.f, 0.f, 0.f, 0.f};
      if (r < g.R && c + 3 < g.L) {
        const float4 v = *reinterpret_cast<const float4*>(sr + (int64_t)r * g.L + c);
        e[0] = v.x; e[1] = v.y; e[2] = v.z; e[3] = v.w;
      } else if (r < g.R) {
        for (int j = 0; j < 4 && c + j < g.L; ++j) e[j] = sr[(int64_t)r * g.L + c + j];
      }
      x.x += e[0]; x.y += e[1]; x.z += e[2]; x.w += e[3];
    }
    x.x *= sign; x.y *= sign; x.z *= sign; x.w *= sign;
    tile[k][q] = x.x;
    tile[k][q + 1] = x.y;
    tile[k][q + 2] = x.z;
    tile[k][q + 3] = x.w;
  }
  __syncthreads();
  if (g.dst) {   // uniform over the block
    T* out = reinterpret_cast<T*>(g.dst) + inst * g.dst_inst;
    for (int k = t >> 4; k < 64; k += 16) {
      const int r = r0 + k, c = c0 + q;
      if (r >= g.R) continue;
      const int64_t o = (int64_t)r * g.ld + c;
      if (c + 3 < g.L && (o & 3) == 0) {
        st4<T>(out, o, tile[k][q], tile[k][q + 1], tile[k][q + 2], tile[k][q + 3]);
      } else {
        for (int j = 0; j < 4 && c + j < g.L; ++j) out[o + j] = (T)tile[k][q + j];
      }
    }
  }
  if (g.dstT) {
    T* out = reinterpret_cast<T*>(g.dstT) + inst * g.dstT_inst;
    for (int k = t >> 4; k < 64; k += 16) {   // output row = input column c0 + k, elements r0 + q .. + 3
      const int c = c0 + k, r = r0 + q;
      if (c >= g.L) continue;
      const int64_t o = (int64_t)c * g.ldT + r;
      if (r + 3 < g.R && (o & 3) == 0) {
        st4<T>(out, o, tile[q][k], tile[q + 1][k], tile[q + 2][k], tile[q + 3][k]);
      } else {
        for (int j = 0; j < 4 && r + j < g.R; ++j) out[o + j] = (T)tile[q + j][k];
      }
    }
  }
}

// Momentum reverse of one chunk (see MomBwdArgs): each block a fixed range
// of one instance's nmat * dh floats, its share of <dM', M> in a fixed order.
__global__ __launch_bounds__(256) void k_mom_bwd(const MomBwdArgs a) {
  __shared__ float red[4];
  const int inst = blockIdx.x / a.nblk, b = blockIdx.x - inst * a.nblk;
  const int64_t n4 = a.nmat * a.dh / 4, per = (n4 + a.nblk - 1) / a.nblk;
  const int64_t e0 = b * per, e1 = e0 + per < n4 ? e0 + per : n4;
  const float bb = a.bbar[inst * a.bbar_inst];
  float dot = 0.0f;
  for (int64_t e = e0 + threadIdx.x; e < e1; e += 256) {
    const int j = (int)((4 * e) / a.dh);
    const int64_t off = inst * a.dh + 4 * e - j * a.dh;
    float4* u = reinterpret_cast<float4*>(a.U + inst * a.nmat * a.dh) + e;
    float4* r = reinterpret_cast<float4*>(a.R[j] + off);
    const float4 m = *reinterpret_cast<const float4*>(a.M[j] + off);
    const float4 uu = *u, rr = *r;
    const float4 t = make_float4(rr.x - uu.x, rr.y - uu.y, rr.z - uu.z, rr.w - uu.w);   // dM'
    dot += t.x * m.x + t.y * m.y + t.z * m.z + t.w * m.w;
    *u = make_float4(-t.x, -t.y, -t.z, -t.w);
    *r = make_float4(bb * t.x, bb * t.y, bb * t.z, bb * t.w);
  }
  dot = wave_sum(dot);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = dot;
  __syncthreads();
  if (threadIdx.x == 0) a.part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// dbeta of a chunk's tokens: one block per instance, the partials summed in order.
__global__ __launch_bounds__(256) void k_mom_dbeta(const float* part, int nblk, float* dbeta, int64_t n_kv,
                                                   int64_t n) {
  __shared__ float tot;
  if (threadIdx.x == 0) {
    float s = 0.0f;
    for (int b = 0; b < nblk; ++b) s += part[(int64_t)blockIdx.x * nblk + b];
    tot = s / (float)n;
  }
  __syncthreads();
  for (int64_t t = threadIdx.x; t < n; t += 256) dbeta[(int64_t)blockIdx.x * n_kv + t] = tot;
}

// M' = bbar M - sum P per instance (grid stride over float4s).
__global__ __launch_bounds__(256) void k_mom_adv(const float* M, const float* bbar, int64_t bbar_inst, const PartSet P,
                                                 float* Mout, int BH, int64_t dh) {
  const int64_t n4 = dh >> 2, total = (int64_t)BH * n4;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < total; x += (int64_t)gridDim.x * 256) {
    const int64_t inst = x / n4;
    const int i = (int)(x - inst * n4);
    const float bb = bbar[inst * bbar_inst];
    const float4 m = reinterpret_cast<const float4*>(M + inst * dh)[i];
    float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
    add_set(P, inst, 0, i, g);
    reinterpret_cast<float4*>(Mout + inst * dh)[i] = make_float4(bb * m.x - g.x, bb * m.y - g.y, bb * m.z - g.z,
                                                                 bb * m.w - g.w);
  }
}

// Sum over one slot of x * y, one workgroup per slot (a fixed reduction
// order, so repeated calls agree bit for bit).
// Sum over one slot of x * y in two passes of fixed order: kDotBlocks
// workgroups per slot each sum a contiguous range of float4s into part,
// then one wave per slot adds the slot's partials in order.
constexpr int kDotBlocks = 32;
__global__ __launch_bounds__(256) void k_slot_dot_part(const float* x, const float* y, int64_t len, float* part) {
  __shared__ float red[4];
  const int64_t slot = blockIdx.x / kDotBlocks;
  const int b = (int)(blockIdx.x - slot * kDotBlocks);
  const int64_t n4 = len >> 2, per = (n4 + kDotBlocks - 1) / kDotBlocks;
  const int64_t i0 = b * per, i1 = i0 + per < n4 ? i0 + per : n4;
  const float4* x4 = reinterpret_cast<const float4*>(x + slot * len);
  const float4* y4 = reinterpret_cast<const float4*>(y + slot * len);
  float acc = 0.0f;
  for (int64_t i = i0 + threadIdx.x; i < i1; i += 256) {
    const float4 a = x4[i], c = y4[i];
    acc += a.x * c.x + a.y * c.y + a.z * c.z + a.w * c.w;
  }
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(64) void k_slot_dot_sum(const float* part, float* out) {
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int b = 0; b < kDotBlocks; ++b) t += part[(int64_t)blockIdx.x * kDotBlocks + b];
    out[blockIdx.x] = t;
  }
}

// Elementwise steps of the Newton-Schulz reverse (see NsLinArgs), grid stride.
__global__ __launch_bounds__(256) void k_ns_lin(const NsLinArgs a) {
  const int64_t n4 = a.len >> 2, total = (int64_t)a.S * n4;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += (int64_t)gridDim.x * 256) {
    const int64_t slot = q / n4;
    const float4 x = reinterpret_cast<const float4*>(a.x)[q];
    float4 r;
    if (a.mode == 0) {
      const float f = 1.0f / (sqrtf(a.sc[slot]) + a.eps);
      r = make_float4(x.x * f, x.y * f, x.z * f, x.w * f);
    } else if (a.mode == 1) {
      r = make_float4(a.a * x.x, a.a * x.y, a.a * x.z, a.a * x.w);
      if (a.p1) {
        const float4 p = reinterpret_cast<const float4*>(a.p1)[q];
        r.x += p.x; r.y += p.y; r.z += p.z; r.w += p.w;
      }
      if (a.p2) {
        const float4 p = reinterpret_cast<const float4*>(a.p2)[q];
        r.x += p.x; r.y += p.y; r.z += p.z; r.w += p.w;
      }
    } else {
      const float nrm = sqrtf(a.sc[slot]), se = nrm + a.eps;
      const float f = 1.0f / se, gf = a.sc2[slot] / (se * se * nrm);
      const float4 y = reinterpret_cast<const float4*>(a.y)[q];
      r = make_float4(x.x * f - gf * y.x, x.y * f - gf * y.y, x.z * f - gf * y.z, x.w * f - gf * y.w);
    }
    if (a.out32) reinterpret_cast<float4*>(a.out32)[q] = r;
    if (a.out16) st4<_Float16>(a.out16, 4 * q, r.x, r.y, r.z, r.w);
    if (a.outc32) reinterpret_cast<float4*>(a.outc32)[q] = r;
  }
}

// out = alpha X + beta (Y + Y^T) per slot of fp16 [m x m] matrices: one
// 32 x 32 output tile per block, Y's mirror tile through LDS.
// 64 x 64 tiles, each row segment moved as 16-byte vectors of 8 halves (m is
// a multiple of 8, so a vector lies wholly inside or outside the matrix);
// the mirror tile goes through LDS.
__global__ __launch_bounds__(256) void k_sym(const _Float16* X, float alpha, const _Float16* Y, float beta,
                                             _Float16* out, int m, int tiles) {
  typedef __attribute__((ext_vector_type(8))) _Float16 h8;
  __shared__ float mir[64][65];
  const int per = tiles * tiles;
  const int64_t slot = blockIdx.x / per;
  const int rest = blockIdx.x - (int)slot * per;
  const int r0 = (rest / tiles) * 64, c0 = (rest % tiles) * 64;
  const int64_t base = slot * (int64_t)m * m;
  const int tv = threadIdx.x & 7, ty = threadIdx.x >> 3;   // 8 vectors per 64-wide row, 32 rows per pass
  for (int k = ty; k < 64; k += 32) {   // mirror tile: mir[k][j] = Y[c0 + k][r0 + j]
    const int r = c0 + k, c = r0 + 8 * tv;
    h8 y = {};
    if (r < m && c < m) y = *reinterpret_cast<const h8*>(Y + base + (int64_t)r * m + c);
#pragma unroll
    for (int j = 0; j < 8; ++j) mir[k][8 * tv + j] = (float)y[j];
  }
  __syncthreads();
  for (int k = ty; k < 64; k += 32) {
    const int r = r0 + k, c = c0 + 8 * tv;
    if (r >= m || c >= m) continue;
    const int64_t o = base + (int64_t)r * m + c;
    const h8 y = *reinterpret_cast<const h8*>(Y + o);
    h8 x = {};
    if (X) x = *reinterpret_cast<const h8*>(X + o);
    h8 v;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float t = beta * ((float)y[j] + mir[8 * tv + j][k]);
      if (X) t += alpha * (float)x[j];
      v[j] = (_Float16)t;
    }
    *reinterpret_cast<h8*>(out + o) = v;
  }
}

// The fp32 form of k_sym: 64 x 64 tiles, float4 vectors (m a multiple of 4).
__global__ __launch_bounds__(256) void k_sym32(const float* X, float alpha, const float* Y, float beta, float* out,
                                               int m, int tiles) {
  __shared__ float mir[64][65];
  const int per = tiles * tiles;
  const int64_t slot = blockIdx.x / per;
  const int rest = blockIdx.x - (int)slot * per;
  const int r0 = (rest / tiles) * 64, c0 = (rest % tiles) * 64;
  const int64_t base = slot * (int64_t)m * m;
  const int tv = threadIdx.x & 15, ty = threadIdx.x >> 4;   // 16 vectors per 64-wide row, 16 rows per pass
  for (int k = ty; k < 64; k += 16) {   // mirror tile: mir[k][j] = Y[c0 + k][r0 + j]
    const int r = c0 + k, c = r0 + 4 * tv;
    float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < m && c < m) y = *reinterpret_cast<const float4*>(Y + base + (int64_t)r * m + c);
    mir[k][4 * tv] = y.x;
    mir[k][4 * tv + 1] = y.y;
    mir[k][4 * tv + 2] = y.z;
    mir[k][4 * tv + 3] = y.w;
  }
  __syncthreads();
  for (int k = ty; k < 64; k += 16) {
    const int r = r0 + k, c = c0 + 4 * tv;
    if (r >= m || c >= m) continue;
    const int64_t o = base + (int64_t)r * m + c;
    const float4 y = *reinterpret_cast<const float4*>(Y + o);
    float4 v = make_float4(beta * (y.x + mir[4 * tv][k]), beta * (y.y + mir[4 * tv + 1][k]),
                           beta * (y.z + mir[4 * tv + 2][k]), beta * (y.w + mir[4 * tv + 3][k]));
    if (X) {
      const float4 x = *reinterpret_cast<const float4*>(X + o);
      v.x += alpha * x.x;
      v.y += alpha * x.y;
      v.z += alpha * x.z;
      v.w += alpha * x.w;
    }
    *reinterpret_cast<float4*>(out + o) = v;
  }
}

// G = base + the sets, grid stride over BH x RL / 4 float4s.
__global__ __launch_bounds__(256) void k_accum(float* G, int64_t g_inst, const float* init, int64_t i_inst, int mode,
                                               const PartSet s0, const PartSet s1, int BH, int64_t RL) {
  const int64_t per = RL >> 2, total = (int64_t)BH * per;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < total; x += (int64_t)gridDim.x * 256) {
    const int64_t inst = x / per;
    const int i = (int)(x - inst * per);
    float4* g = reinterpret_cast<float4*>(G + inst * g_inst) + i;
    float4 acc = mode == 0 ? make_float4(0.f, 0.f, 0.f, 0.f)
                           : (mode == 1 ? reinterpret_cast<const float4*>(init + inst * i_inst)[i] : *g);
    add_set(s0, inst, 0, i, acc);
    add_set(s1, inst, 0, i, acc);
    *g = acc;
  }
}

// Linear fast weight, one wave per key token t of a chunk (grid stride over
// BH x n tokens). On entry dv holds Y = K Uh^T (rows t); it leaves as
// dv_t = eta_t Y_t, with deta_t = v_t . Y_t (= v_t^T Uh k_t).
template <typename T>
__global__ __launch_bounds__(256) void k_lin_tokens(const T* V, const float* eta, T* dv, float* deta, int BH,
                                                    int64_t n, int d, int64_t tok_inst, int64_t eta_inst) {
  const int lane = threadIdx.x & 63;
  const int64_t total = (int64_t)BH * n;
  for (int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wave < total; wave += (int64_t)gridDim.x * 4) {
    const int64_t inst = wave / n, t = wave - inst * n;
    const int64_t o = inst * tok_inst + t * d;
    const float e = eta[inst * eta_inst + t];
    float dot = 0.0f;
    for (int c = 4 * lane; c < d; c += 256) {
      float y[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        y[q] = (float)dv[o + c + q];
        dot += (float)V[o + c + q] * y[q];
      }
      st4<T>(dv, o + c, e * y[0], e * y[1], e * y[2], e * y[3]);
    }
    dot = wave_sum(dot);
    if (lane == 0) deta[inst * eta_inst + t] = dot;
  }
}

template <typename T>
__device__ __forceinline__ void ld4(const void* base, int64_t idx, float* v) {
  const T* p = reinterpret_cast<const T*>(base) + idx;
  if constexpr (sizeof(T) == 2) {
    typedef __attribute__((ext_vector_type(4))) T t4;
    const t4 x = *reinterpret_cast<const t4*>(p);
    v[0] = (float)x[0]; v[1] = (float)x[1]; v[2] = (float)x[2]; v[3] = (float)x[3];
  } else {
    const float4 x = *reinterpret_cast<const float4*>(p);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  }
}

// SwiGLU chunk-gradient reverse, one wave per key token (grid stride). With
// S = SiLU(Z1), S1 = SiLU'(Z1), S2 = SiLU''(Z1), A = S Z3 and the token's
// rates e1, e2, e3 of W1, W2, W3 (one rate: all three the same):
//   dA  = e2 Y2,  dC = e3 X3 S + e1 X1 Z3 S1,  dZ3 = e1 X1 C S1 + dA S,
//   dZ1 = (e3 X3 C + dA Z3) S1 + e1 X1 C Z3 S2,  R3 = e3 C S,  R1 = e1 C Z3 S1,
//   and, summed over the hidden units, de1 = X1 C Z3 S1, de2 = A Y2,
//   de3 = X3 C S (one rate: deta = their sum).
template <typename T>
__global__ __launch_bounds__(256) void k_swiglu_rows(const SwigluRowsArgs a) {
  const int lane = threadIdx.x & 63;
  const int h = a.h;
  const bool per_matrix = a.eta_cols == 3;
  const int64_t total = (int64_t)a.BH * a.n;
  for (int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wave < total; wave += (int64_t)gridDim.x * 4) {
    const int64_t inst = wave / a.n, t = wave - inst * a.n;
    const int64_t io = inst * a.in_inst + t * h, zo = inst * (a.z_inst ? a.z_inst : a.in_inst) + t * h;
    const int64_t ko = inst * a.pk_inst + t * 4 * h, vo = inst * a.pv_inst + t * 2 * h;
    const int64_t eo = (inst * a.eta_inst + t) * a.eta_cols;
    const float e1 = a.eta[eo];
    const float e2 = per_matrix ? a.eta[eo + 1] : e1, e3 = per_matrix ? a.eta[eo + 2] : e1;
    float d1 = 0.0f, d2 = 0.0f, d3 = 0.0f;
    for (int j = 4 * lane; j < h; j += 256) {
      float z1[4], z3[4], c[4], x1[4], x3[4], y2[4];
      ld4<T>(a.Z1, zo + j, z1);
      ld4<T>(a.Z3, zo + j, z3);
      ld4<T>(a.C, zo + j, c);
      ld4<T>(a.X1, io + j, x1);
      ld4<T>(a.X3, io + j, x3);
      ld4<T>(a.Y2, io + j, y2);
      float r3[4], r1[4], dz1[4], dz3[4], ea[4], dc[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float sg = sigmoidf_fast(z1[q]);
        const float S = z1[q] * sg, S1 = sg + z1[q] * sg * (1.0f - sg);
        const float S2 = sg * (1.0f - sg) * (2.0f + z1[q] * (1.0f - 2.0f * sg));
        const float A = S * z3[q], dA = e2 * y2[q];
        const float t1 = x1[q] * c[q] * z3[q] * S1, t3 = x3[q] * c[q] * S;
        dc[q] = e3 * x3[q] * S + e1 * x1[q] * z3[q] * S1;
        dz3[q] = e1 * x1[q] * c[q] * S1 + dA * S;
        dz1[q] = (e3 * x3[q] * c[q] + dA * z3[q]) * S1 + e1 * x1[q] * c[q] * z3[q] * S2;
        r3[q] = e3 * c[q] * S;
        r1[q] = e1 * c[q] * z3[q] * S1;
        ea[q] = e2 * A;
        d1 += t1;
        d2 += A * y2[q];
        d3 += t3;
      }
      st4<T>(a.Pk, ko + j, r3[0], r3[1], r3[2], r3[3]);
      st4<T>(a.Pk, ko + h + j, r1[0], r1[1], r1[2], r1[3]);
      st4<T>(a.Pk, ko + 2 * h + j, dz1[0], dz1[1], dz1[2], dz1[3]);
      st4<T>(a.Pk, ko + 3 * h + j, dz3[0], dz3[1], dz3[2], dz3[3]);
      st4<T>(a.Pv, vo + j, ea[0], ea[1], ea[2], ea[3]);
      st4<T>(a.Pv, vo + h + j, dc[0], dc[1], dc[2], dc[3]);
    }
    if (per_matrix) {
      d1 = wave_sum(d1);
      d2 = wave_sum(d2);
      d3 = wave_sum(d3);
      if (lane == 0) {
        a.deta[eo] = d1;
        a.deta[eo + 1] = d2;
        a.deta[eo + 2] = d3;
      }
    } else {
      const float dsum = wave_sum(d2 + d3 + d1);
      if (lane == 0) a.deta[eo] = dsum;
    }
  }
}

// SwiGLU apply reverse, one wave per query token (grid stride):
// Hq = SiLU(Zq1) Zq3, dZq3 = Dh SiLU(Zq1), dZq1 = Dh Zq3 SiLU'(Zq1).
template <typename T>
__global__ __launch_bounds__(256) void k_swiglu_apply_rows(const T* Z1, const T* Z3, const T* Dh, int64_t in_inst, T* Pq,
                                                           int64_t pq_inst, T* Hq, int64_t hq_inst, int BH, int64_t n,
                                                           int h) {
  const int lane = threadIdx.x & 63;
  const int64_t total = (int64_t)BH * n;
  for (int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wave < total; wave += (int64_t)gridDim.x * 4) {
    const int64_t inst = wave / n, t = wave - inst * n;
    const int64_t io = inst * in_inst + t * h, po = inst * pq_inst + t * 2 * h, ho = inst * hq_inst + t * h;
    for (int j = 4 * lane; j < h; j += 256) {
      float z1[4], z3[4], dh[4], d1[4], d3[4], hq[4];
      ld4<T>(Z1, io + j, z1);
      ld4<T>(Z3, io + j, z3);
      ld4<T>(Dh, io + j, dh);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float sg = sigmoidf_fast(z1[q]);
        const float S = z1[q] * sg, S1 = sg + z1[q] * sg * (1.0f - sg);
        hq[q] = S * z3[q];
        d3[q] = dh[q] * S;
        d1[q] = dh[q] * z3[q] * S1;
      }
      st4<T>(Pq, po + j, d1[0], d1[1], d1[2], d1[3]);
      st4<T>(Pq, po + h + j, d3[0], d3[1], d3[2], d3[3]);
      st4<T>(Hq, ho + j, hq[0], hq[1], hq[2], hq[3]);
    }
  }
}

// x[i * inst + off + j] = 0 for j < count, every instance i (grid stride).
__global__ __launch_bounds__(256) void k_zero_f32(float* x, int64_t inst, int64_t off, int64_t count, int64_t total) {
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int64_t i = t / count;
    x[i * inst + off + (t - i * count)] = 0.0f;
  }
}

// Rows [r0, r1) of every instance of a row-major [BH, n, d] output set to zero
// (tokens that no apply segment of a schedule covers): nvec 16-byte vectors
// per instance, grid-stride over all instances.
__global__ __launch_bounds__(256) void k_zero_rows(uint8_t* out, int64_t inst_bytes, int64_t off, int64_t nvec,
                                                   int64_t total) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t inst = i / nvec, j = i - inst * nvec;
    reinterpret_cast<u32x4_t*>(out + inst * inst_bytes + off)[j] = u32x4_t{0u, 0u, 0u, 0u};
  }
}

}  // namespace

// ===========================================================================
// Host-visible shapes and launchers

TileShape fwd_tile(int kind, bool io_bf16, bool narrow) {
  if (io_bf16 && narrow) return TileShape{KApplyN16::ROWS_A, KApplyN16::ROWS_B, KApplyN16::THREADS};
  if (io_bf16) return kind == FWD_APPLY ? TileShape{KApply16::ROWS_A, KApply16::ROWS_B, KApply16::THREADS}
                                        : TileShape{KApply16::ROWS_A, KApply16::ROWS_B, KApply16::THREADS};
  return kind == FWD_APPLY ? TileShape{KApply32::ROWS_A, KApply32::ROWS_B, KApply32::THREADS}
                           : TileShape{KUpdate32::ROWS_A, KUpdate32::ROWS_B, KUpdate32::THREADS};
}

TileShape bwd_tile(int kind, bool io_bf16, bool narrow) {
  if (io_bf16 && narrow) {
    if (kind == BWD_OUT) return TileShape{KOutN16::ROWS_A, KOutN16::ROWS_B, KOutN16::THREADS};
    if (kind == BWD_GRAD13) return TileShape{KGrad13N16::ROWS_A, KGrad13N16::ROWS_B, KGrad13N16::THREADS};
    return TileShape{KGrad2N16::ROWS_A, KGrad2N16::ROWS_B, KGrad2N16::THREADS};
  }
  if (io_bf16) {
    if (kind == BWD_OUT) return TileShape{KOut16::ROWS_A, KOut16::ROWS_B, KOut16::THREADS};
    if (kind == BWD_GRAD13) return TileShape{KGrad13_16::ROWS_A, KGrad13_16::ROWS_B, KGrad13_16::THREADS};
    return TileShape{KGrad2_16::ROWS_A, KGrad2_16::ROWS_B, KGrad2_16::THREADS};
  }
  if (kind == BWD_OUT) return TileShape{KOut32::ROWS_A, KOut32::ROWS_B, KOut32::THREADS};
  if (kind == BWD_GRAD13) return TileShape{KGrad13_32::ROWS_A, KGrad13_32::ROWS_B, KGrad13_32::THREADS};
  return TileShape{KGrad2_32::ROWS_A, KGrad2_32::ROWS_B, KGrad2_32::THREADS};
}

TileShape grad_upd_tile() { return TileShape{KGradU16::ROWS_A, KGradU16::ROWS_B, KGradU16::THREADS}; }

TileShape ns_tile(bool fp16, bool big) {
  if (fp16 && big) return TileShape{KNsK16B::ROWS_A, KNsK16B::ROWS_B, KNsK16B::THREADS};
  if (fp16) return TileShape{KNsK16S::ROWS_A, KNsK16S::ROWS_B, KNsK16S::THREADS};
  return TileShape{KNsK32::ROWS_A, KNsK32::ROWS_B, KNsK32::THREADS};
}

TileShape ns_final_tile() { return TileShape{KNsRow16::ROWS_A, KNsRow16::ROWS_B, KNsRow16::THREADS}; }

hipError_t launch_ns_final(const NsFinalArgs& a, hipStream_t s) {
  if (a.nblocks <= 0) return hipSuccess;
  k_ns_final<<<a.nblocks, KNsRow16::THREADS, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_ns(const NsArgs& a, bool fp16, bool big, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  if (fp16 && big) k_ns<_Float16, true><<<a.total_blocks, KNsK16B::THREADS, 0, s>>>(a);
  else if (fp16) k_ns<_Float16, false><<<a.total_blocks, KNsK16S::THREADS, 0, s>>>(a);
  else k_ns<float, false><<<a.total_blocks, KNsK32::THREADS, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_ns_fused(const NsFusedArgs& a, hipStream_t s) {
  if (a.nblocks <= 0) return hipSuccess;
  if (a.rows > a.cols) k_ns_fused<true><<<a.nblocks, 512, 0, s>>>(a);
  else k_ns_fused<false><<<a.nblocks, 512, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_ns_fused_pair(const NsFusedArgs& a0, const NsFusedArgs& a1, hipStream_t s) {
  if (a0.nblocks + a1.nblocks <= 0) return hipSuccess;
  const int64_t blocks = (int64_t)a0.nblocks + a1.nblocks;
  // the two groups are transposes of each other's shape: at most one is tall
  if (a0.rows > a0.cols) k_ns_fused_pair<true, false><<<(unsigned)blocks, 512, 0, s>>>(a0, a1);
  else if (a1.rows > a1.cols) k_ns_fused_pair<false, true><<<(unsigned)blocks, 512, 0, s>>>(a0, a1);
  else k_ns_fused_pair<false, false><<<(unsigned)blocks, 512, 0, s>>>(a0, a1);
  return hipGetLastError();
}

hipError_t launch_ns_fused_pair_out(const NsFusedArgs& a0, const NsFusedArgs& a1, const BwdArgs& out,
                                    hipStream_t s) {
  const int64_t blocks = (int64_t)a0.nblocks + a1.nblocks + out.total_blocks;
  if (blocks <= 0) return hipSuccess;
  if (!out.narrow || out.nseg != 1 || out.seg[0].kind != BWD_OUT) return hipErrorInvalidValue;
  if (a0.rows > a0.cols) k_ns_fused_pair_out<true, false><<<(unsigned)blocks, 512, 0, s>>>(a0, a1, out);
  else if (a1.rows > a1.cols) k_ns_fused_pair_out<false, true><<<(unsigned)blocks, 512, 0, s>>>(a0, a1, out);
  else k_ns_fused_pair_out<false, false><<<(unsigned)blocks, 512, 0, s>>>(a0, a1, out);
  return hipGetLastError();
}

hipError_t launch_ns_prep(const NsPrepArgs& a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.nslots * a.blocks_per_slot;
  if (blocks <= 0) return hipSuccess;
  k_ns_prep<<<(unsigned)blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_ns_scale(const NsPrepArgs& a, void* Yb, bool fp16, float eps, hipStream_t s) {
  const int64_t blocks = (int64_t)a.nslots * a.blocks_per_slot;
  if (blocks <= 0) return hipSuccess;
  if (fp16) k_ns_scale<_Float16><<<(unsigned)blocks, 256, 0, s>>>(a, Yb, eps);
  else k_ns_scale<float><<<(unsigned)blocks, 256, 0, s>>>(a, Yb, eps);
  return hipGetLastError();
}

hipError_t launch_zero_rows(void* out, int BH, int64_t row_bytes, int64_t rows, int64_t r0, int64_t r1,
                            hipStream_t s) {
  const int64_t nvec = (r1 - r0) * row_bytes / 16, total = nvec * BH;
  if (nvec <= 0 || BH <= 0) return hipSuccess;
  const int64_t need = (total + 255) / 256, blocks = need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20);
  k_zero_rows<<<(unsigned)blocks, 256, 0, s>>>(reinterpret_cast<uint8_t*>(out), rows * row_bytes, r0 * row_bytes,
                                               nvec, total);
  return hipGetLastError();
}

hipError_t launch_zero_f32(float* x, int BH, int64_t inst, int64_t off, int64_t count, hipStream_t s) {
  const int64_t total = (int64_t)BH * count;
  if (total <= 0) return hipSuccess;
  const int64_t need = (total + 255) / 256, blocks = need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20);
  k_zero_f32<<<(unsigned)blocks, 256, 0, s>>>(x, inst, off, count, total);
  return hipGetLastError();
}

hipError_t launch_beta_mean(const BetaArgs& a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.BH * a.nchunks;
  if (blocks <= 0) return hipSuccess;
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  k_beta_mean<<<(unsigned)blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_fwd(const FwdArgs& a, bool io_bf16, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  bool keep = false;
  for (int i = 0; i < a.nseg; ++i) keep = keep || (a.seg[i].kind == FWD_UPDATE && a.seg[i].keep[0]);
  if (keep) {
    if (io_bf16 && a.narrow) k_fwd_narrow_keep<<<a.total_blocks, KApplyN16::THREADS, 0, s>>>(a);
    else if (io_bf16) k_fwd_keep<__bf16><<<a.total_blocks, KApply16::THREADS, 0, s>>>(a);
    else k_fwd_keep<float><<<a.total_blocks, KApply32::THREADS, 0, s>>>(a);
    return hipGetLastError();
  }
  if (io_bf16 && a.narrow) k_fwd_narrow<<<a.total_blocks, KApplyN16::THREADS, 0, s>>>(a);
  else if (io_bf16) k_fwd<__bf16><<<a.total_blocks, KApply16::THREADS, 0, s>>>(a);
  else k_fwd<float><<<a.total_blocks, KApply32::THREADS, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdArgs& a, bool io_bf16, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  if (io_bf16 && a.narrow) k_bwd<__bf16, true><<<a.total_blocks, KOutN16::THREADS, 0, s>>>(a);
  else if (io_bf16) k_bwd<__bf16, false><<<a.total_blocks, KOut16::THREADS, 0, s>>>(a);
  else k_bwd<float, false><<<a.total_blocks, KOut32::THREADS, 0, s>>>(a);
  return hipGetLastError();
}

template <int NV>
static void launch_update_nv(const UpdArgs& a, bool io_bf16, int blocks, hipStream_t s) {
  if (io_bf16) k_update<__bf16, NV><<<blocks, 256, 0, s>>>(a);
  else k_update<float, NV><<<blocks, 256, 0, s>>>(a);
}

hipError_t launch_update(const UpdArgs& a, bool io_bf16, hipStream_t s) {
  const int blocks = (a.rows_total + 3) / 4;   // a wave per row
  if (blocks <= 0) return hipSuccess;
  const int L = a.d > a.h ? a.d : a.h;        // longest row, floats
  const int per_lane = (L / 4 + 63) / 64;      // float4 vectors per lane
  if (per_lane <= 1) launch_update_nv<1>(a, io_bf16, blocks, s);
  else if (per_lane <= 2) launch_update_nv<2>(a, io_bf16, blocks, s);
  else if (per_lane <= 4) launch_update_nv<4>(a, io_bf16, blocks, s);
  else if (per_lane <= 8) launch_update_nv<8>(a, io_bf16, blocks, s);
  else launch_update_nv<16>(a, io_bf16, blocks, s);
  return hipGetLastError();
}

hipError_t launch_scale_rows(const void* k, const float* eta, void* out, int BH, int64_t n, int d, int64_t k_inst,
                             int64_t eta_inst, int64_t out_inst, bool io_bf16, hipStream_t s) {
  const int64_t total = (int64_t)BH * n * (d / (io_bf16 ? 8 : 4));
  if (total <= 0) return hipSuccess;
  const int64_t need = (total + 255) / 256, blocks = need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20);
  const bool small = total < ((int64_t)1 << 31);
  if (io_bf16) {
    const __bf16* kk = reinterpret_cast<const __bf16*>(k);
    __bf16* oo = reinterpret_cast<__bf16*>(out);
    if (small) k_scale_rows<__bf16, uint32_t><<<(unsigned)blocks, 256, 0, s>>>(kk, eta, oo, n, d, k_inst, eta_inst, out_inst, total);
    else k_scale_rows<__bf16, uint64_t><<<(unsigned)blocks, 256, 0, s>>>(kk, eta, oo, n, d, k_inst, eta_inst, out_inst, total);
  } else {
    const float* kk = reinterpret_cast<const float*>(k);
    float* oo = reinterpret_cast<float*>(out);
    if (small) k_scale_rows<float, uint32_t><<<(unsigned)blocks, 256, 0, s>>>(kk, eta, oo, n, d, k_inst, eta_inst, out_inst, total);
    else k_scale_rows<float, uint64_t><<<(unsigned)blocks, 256, 0, s>>>(kk, eta, oo, n, d, k_inst, eta_inst, out_inst, total);
  }
  return hipGetLastError();
}

hipError_t launch_prep(const float* const W[3], void* const Wb[3], int BH, int d, int h, hipStream_t s) {
  const int64_t n4 = (int64_t)BH * d * h / 4;
  const int64_t blocks = (n4 + 255) / 256;
  if (blocks <= 0) return hipSuccess;
  k_prep<<<(unsigned)blocks, 256, 0, s>>>(W[0], W[1], W[2], reinterpret_cast<__bf16*>(Wb[0]),
                                         reinterpret_cast<__bf16*>(Wb[1]), reinterpret_cast<__bf16*>(Wb[2]), n4);
  return hipGetLastError();
}

// Backward steps between the OUT / GRAD contractions (io_bf16 selects bf16
// operand copies, else fp32).
hipError_t launch_vjp(const VjpArgs* a, int n, bool io_bf16, hipStream_t s) {
  if (n < 1 || n > 3) return hipErrorInvalidValue;
  int Lmax = 0;
  for (int i = 0; i < n; ++i) Lmax = a[i].L > Lmax ? a[i].L : Lmax;
  const int per_lane = (Lmax / 4 + 63) / 64;
  const VjpArgs none{};
  auto go = [&](auto tag, auto nvc) {
    using T = decltype(tag);
    constexpr int NV = decltype(nvc)::value;
    constexpr int RR = vjp_rows<T, NV>();
    int nb[3] = {0, 0, 0};
    for (int i = 0; i < n; ++i) nb[i] = a[i].BH * ((a[i].R + RR - 1) / RR);   // <= 2^20 * 1024 each
    const int64_t blocks = (int64_t)nb[0] + nb[1] + nb[2];
    if (blocks <= 0) return;
    k_vjp<T, NV><<<(unsigned)blocks, 64 * vjp_waves<NV>(), 0, s>>>(a[0], n > 1 ? a[1] : none, n > 2 ? a[2] : none,
                                                                   nb[0], nb[1]);
  };
  auto pick = [&](auto tag) {
    if (per_lane <= 1) go(tag, std::integral_constant<int, 1>{});
    else if (per_lane <= 2) go(tag, std::integral_constant<int, 2>{});
    else if (per_lane <= 4) go(tag, std::integral_constant<int, 4>{});
    else if (per_lane <= 8) go(tag, std::integral_constant<int, 8>{});
    else go(tag, std::integral_constant<int, 16>{});
  };
  if (io_bf16) pick(__bf16{});
  else pick(float{});
  return hipGetLastError();
}

hipError_t launch_copies(const CopySeg* c, int n, int BH, bool io_bf16, hipStream_t s) {
  if (n < 0 || n > kMaxCopies) return hipErrorInvalidValue;
  CopyArgs a{};
  a.n = n;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    a.seg[i] = c[i];
    a.first[i] = (int)total;
    total += (int64_t)BH * ((c[i].R + 63) / 64) * ((c[i].L + 63) / 64);
  }
  // callers keep the sum under 2^31 (one set of weights: under 2^28 each by the descriptor check)
  if (total <= 0) return hipSuccess;
  if (total >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  a.first[n] = (int)total;
  if (io_bf16) k_copies<__bf16><<<(unsigned)total, 256, 0, s>>>(a);
  else k_copies<float><<<(unsigned)total, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_copies_f32(const CopySeg* c, int n, int BH, hipStream_t s) {
  if (n < 0 || n > kMaxCopies) return hipErrorInvalidValue;
  CopyArgs a{};
  a.n = n;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    a.seg[i] = c[i];
    a.first[i] = (int)total;
    total += (int64_t)BH * ((c[i].R + 63) / 64) * ((c[i].L + 63) / 64);
  }
  if (total <= 0) return hipSuccess;
  if (total >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  a.first[n] = (int)total;
  k_copies<float><<<(unsigned)total, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_mom_bwd(const MomBwdArgs& a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.BH * a.nblk;
  if (blocks <= 0) return hipSuccess;
  k_mom_bwd<<<(unsigned)blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_mom_dbeta(const float* part, int nblk, int BH, float* dbeta, int64_t n_kv, int64_t n, hipStream_t s) {
  if (BH <= 0 || n <= 0) return hipSuccess;
  k_mom_dbeta<<<(unsigned)BH, 256, 0, s>>>(part, nblk, dbeta, n_kv, n);
  return hipGetLastError();
}

hipError_t launch_mom_adv(const float* M, const float* bbar, int64_t bbar_inst, PartSet P, float* Mout, int BH,
                          int64_t dh, hipStream_t s) {
  const int64_t need = ((int64_t)BH * (dh / 4) + 255) / 256;
  if (need <= 0) return hipSuccess;
  const int64_t blocks = need < 8192 ? need : 8192;
  k_mom_adv<<<(unsigned)blocks, 256, 0, s>>>(M, bbar, bbar_inst, P, Mout, BH, dh);
  return hipGetLastError();
}

hipError_t launch_bwd_f16(const BwdArgs& a, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  if (a.narrow) k_bwd<_Float16, true><<<a.total_blocks, KOutN16::THREADS, 0, s>>>(a);
  else k_bwd<_Float16, false><<<a.total_blocks, KOut16::THREADS, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_slot_dot(const float* x, const float* y, int S, int64_t len, float* out, float* part,
                           hipStream_t s) {
  if (S <= 0) return hipSuccess;
  if ((int64_t)S * kDotBlocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  k_slot_dot_part<<<(unsigned)(S * kDotBlocks), 256, 0, s>>>(x, y, len, part);
  k_slot_dot_sum<<<(unsigned)S, 64, 0, s>>>(part, out);
  return hipGetLastError();
}

hipError_t launch_ns_lin(const NsLinArgs& a, hipStream_t s) {
  const int64_t need = ((int64_t)a.S * (a.len / 4) + 255) / 256;
  if (need <= 0) return hipSuccess;
  const int64_t blocks = need < 8192 ? need : 8192;
  k_ns_lin<<<(unsigned)blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_sym(const _Float16* X, float alpha, const _Float16* Y, float beta, _Float16* out, int S, int m,
                      hipStream_t s) {
  if (m % 8) return hipErrorInvalidValue;
  const int tiles = (m + 63) / 64;
  const int64_t blocks = (int64_t)S * tiles * tiles;
  if (blocks <= 0) return hipSuccess;
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  k_sym<<<(unsigned)blocks, 256, 0, s>>>(X, alpha, Y, beta, out, m, tiles);
  return hipGetLastError();
}

hipError_t launch_sym32(const float* X, float alpha, const float* Y, float beta, float* out, int S, int m,
                        hipStream_t s) {
  if (m % 4) return hipErrorInvalidValue;
  const int tiles = (m + 63) / 64;
  const int64_t blocks = (int64_t)S * tiles * tiles;
  if (blocks <= 0) return hipSuccess;
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  k_sym32<<<(unsigned)blocks, 256, 0, s>>>(X, alpha, Y, beta, out, m, tiles);
  return hipGetLastError();
}

hipError_t launch_accum(float* G, int64_t g_inst, const float* init, int64_t i_inst, int mode, PartSet s0, PartSet s1,
                        int BH, int64_t RL, hipStream_t s) {
  const int64_t need = ((int64_t)BH * (RL / 4) + 255) / 256;
  if (need <= 0) return hipSuccess;
  const int64_t blocks = need < 4096 ? need : 4096;
  k_accum<<<(unsigned)blocks, 256, 0, s>>>(G, g_inst, init, i_inst, mode, s0, s1, BH, RL);
  return hipGetLastError();
}

hipError_t launch_lin_tokens(const void* V, const float* eta, void* dv, float* deta, int BH, int64_t n, int d,
                             int64_t tok_inst, int64_t eta_inst, bool io_bf16, hipStream_t s) {
  const int64_t rows = (int64_t)BH * n;
  if (rows <= 0) return hipSuccess;
  const int64_t need = (rows + 3) / 4;
  const unsigned blocks = (unsigned)(need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20));
  if (io_bf16)
    k_lin_tokens<__bf16><<<blocks, 256, 0, s>>>(reinterpret_cast<const __bf16*>(V), eta, reinterpret_cast<__bf16*>(dv),
                                                deta, BH, n, d, tok_inst, eta_inst);
  else
    k_lin_tokens<float><<<blocks, 256, 0, s>>>(reinterpret_cast<const float*>(V), eta, reinterpret_cast<float*>(dv),
                                               deta, BH, n, d, tok_inst, eta_inst);
  return hipGetLastError();
}

hipError_t launch_swiglu_rows(const SwigluRowsArgs& a, bool io_bf16, hipStream_t s) {
  const int64_t rows = (int64_t)a.BH * a.n;
  if (rows <= 0) return hipSuccess;
  const int64_t need = (rows + 3) / 4;
  const unsigned blocks = (unsigned)(need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20));
  if (io_bf16) k_swiglu_rows<__bf16><<<blocks, 256, 0, s>>>(a);
  else k_swiglu_rows<float><<<blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_swiglu_apply_rows(const void* Z1, const void* Z3, const void* Dh, int64_t in_inst, void* Pq,
                                    int64_t pq_inst, void* Hq, int64_t hq_inst, int BH, int64_t n, int h, bool io_bf16,
                                    hipStream_t s) {
  const int64_t rows = (int64_t)BH * n;
  if (rows <= 0) return hipSuccess;
  const int64_t need = (rows + 3) / 4;
  const unsigned blocks = (unsigned)(need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20));
  auto go = [&](auto tag) {
    using T = decltype(tag);
    k_swiglu_apply_rows<T><<<blocks, 256, 0, s>>>(reinterpret_cast<const T*>(Z1), reinterpret_cast<const T*>(Z3),
                                                  reinterpret_cast<const T*>(Dh), in_inst, reinterpret_cast<T*>(Pq),
                                                  pq_inst, reinterpret_cast<T*>(Hq), hq_inst, BH, n, h);
  };
  if (io_bf16) go(__bf16{});
  else go(float{});
  return hipGetLastError();
}

}  // namespace lact
