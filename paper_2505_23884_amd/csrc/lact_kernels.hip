// gfx950 kernels of the LaCT fast-weight layer forward.
//
// Every contraction of the path is one 128 x 128 output tile per workgroup
// (256 threads = 4 waves, each wave a 64 x 64 quarter built from 2 x 2
// v_mfma_f32_32x32x16_bf16 blocks, or 32x32x2_f32 in fp32 mode), with fp32
// accumulation and a fused epilogue per kind:
//
//   FWD_APPLY   Z = Q W1^T, Q W3^T          -> hidden SiLU(Z1) o Z3       (apply, §3.1 SwiGLU eq.)
//   FWD_UPDATE  Z = K W1^T, K W3^T, D = V W2 -> eta*hidden, eta*dz1, eta*dz3
//               the key forward and the backward to the hidden units of
//               grad sum_i eta_i (-f_W(k_i)^T v_i)               (§3.1 loss and chunk-gradient eqs.)
//   BWD_OUT     O = hidden W2^T                                    (apply, second matmul)
//   BWD_GRAD13  P1 = (eta dz1)^T K,  P3 = (eta dz3)^T K             (gradient matmuls, -g1, -g3)
//   BWD_GRAD2   P2 = V^T (eta hidden)                              (-g2)
//
// Operands live in HBM either K-contiguous ("kmajor", row-major [rows x K])
// or row-contiguous ("mn", row-major [K x rows], the token-major layout of
// the gradient contractions). Both are staged through LDS as 128 rows x 64
// bytes (32 bf16 or 16 fp32 of K) per operand, double-buffered; mn operands
// are transposed in registers on the way (4 K rows x 8 or 4 elements per
// thread) so that every MFMA fragment is one 16-byte LDS read.
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
constexpr int kTileBytes = kTile * kRowBytes;   // one operand tile in LDS

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

// LDS byte offset of 16-byte chunk `chunk` (0..3) of tile row `row`. The XOR
// keeps the 16 (or 8) lanes that read one MFMA fragment column on distinct
// banks both for a 64-bank and a 32-bank LDS.
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * kRowBytes + ((chunk ^ (((row >> 1) ^ (row >> 3)) & 3)) << 4);
}

// Row permutation of mn-operand tiles: the transposing store writes 8 (bf16)
// or 4 (fp32) rows per thread; rotating rows by the thread's row block puts
// the lanes of one store instruction on distinct bank groups.
template <typename T>
__device__ __forceinline__ int mn_row(int r) {
  if constexpr (sizeof(T) == 2) return r ^ ((r >> 3) & 3);
  else return r ^ ((r >> 2) & 3);
}

__device__ __forceinline__ int xcd_remap(int bid, int n) {
  // Workgroups are dispatched round-robin over the 8 XCDs; give every XCD a
  // contiguous range of logical tiles so neighbours share its L2.
  const int x = bid & 7, idx = bid >> 3, per = n >> 3, rem = n & 7;
  return x * per + (x < rem ? x : rem) + idx;
}

// One operand restricted to the current output tile.
struct View {
  const uint8_t* p;   // element (tile row 0, k 0)
  int64_t ld_b;       // bytes between rows (kmajor) or between K rows (mn)
  int64_t nrows;      // valid rows from tile row 0
  int64_t nk;         // valid K from k 0
};

template <typename T>
__device__ __forceinline__ void gload_k(u32x4_t (&r)[4], const View& v, int64_t k0) {
  constexpr int E = Tr<T>::E;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = threadIdx.x + i * kThreads;
    const int row = q >> 2, c = q & 3;
    const int64_t k = k0 + c * E;
    u32x4_t x = {0u, 0u, 0u, 0u};
    if (row < v.nrows && k < v.nk)
      x = *reinterpret_cast<const u32x4_t*>(v.p + row * v.ld_b + k * (int64_t)sizeof(T));
    r[i] = x;
  }
}

template <typename T>
__device__ __forceinline__ void sstore_k(uint8_t* tile, const u32x4_t (&r)[4]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = threadIdx.x + i * kThreads;
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

template <typename T>
__device__ __forceinline__ void sstore_mn(uint8_t* tile, const u32x4_t (&r)[4], int tt) {
  if constexpr (sizeof(T) == 2) {
    const int kg = tt & 7, mb = tt >> 3;
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const uint32_t x0 = r[0][m >> 1], x1 = r[1][m >> 1], x2 = r[2][m >> 1], x3 = r[3][m >> 1];
      uint32_t lo, hi;
      if (m & 1) {
        lo = (x0 >> 16) | (x1 & 0xFFFF0000u);
        hi = (x2 >> 16) | (x3 & 0xFFFF0000u);
      } else {
        lo = (x0 & 0xFFFFu) | (x1 << 16);
        hi = (x2 & 0xFFFFu) | (x3 << 16);
      }
      const int row = mn_row<T>(mb * 8 + m);
      *reinterpret_cast<u32x2_t*>(tile + lds_off(row, kg >> 1) + ((kg & 1) << 3)) = u32x2_t{lo, hi};
    }
  } else {
    const int kg = tt & 3, mb = tt >> 2;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int row = mn_row<T>(mb * 4 + m);
      *reinterpret_cast<u32x4_t*>(tile + lds_off(row, kg)) = u32x4_t{r[0][m], r[1][m], r[2][m], r[3][m]};
    }
  }
}

template <typename T>
__device__ __forceinline__ u32x4_t frag(const uint8_t* tile, int row, int chunk, bool mn) {
  const int pr = mn ? mn_row<T>(row) : row;
  return *reinterpret_cast<const u32x4_t*>(tile + lds_off(pr, chunk));
}

// ---------------------------------------------------------------------------
// Contraction kinds: operands 0..NA-1 are A (tile rows = output rows),
// NA..NA+NB-1 are B (tile rows = output columns); accumulator p multiplies
// A[pa(p)] by B[pb(p)]. Bit o of MN marks operand o as row-contiguous.
template <int NA_, int NB_, int NACC_, uint32_t MN_>
struct KindBase {
  static constexpr int NA = NA_, NB = NB_, NACC = NACC_, NOPS = NA_ + NB_;
  static constexpr uint32_t MN = MN_;
  static constexpr bool is_mn(int o) { return (MN >> o) & 1u; }
  // which half of the block (threads 0-127 / 128-255) loads mn operand o
  static constexpr int mn_half(int o) { return __builtin_popcount(MN & ((1u << o) - 1u)) & 1; }
};
struct KApply : KindBase<1, 2, 2, 0u> {
  static constexpr int NSTAGE = 4;
  static constexpr int pa(int) { return 0; }
  static constexpr int pb(int p) { return p; }
};
struct KUpdate : KindBase<2, 3, 3, 1u << 4> {     // W2 (operand 4) is read transposed
  static constexpr int NSTAGE = 3;
  static constexpr int pa(int p) { return p == 2 ? 1 : 0; }
  static constexpr int pb(int p) { return p; }
};
struct KOut : KindBase<1, 1, 1, 0u> {
  static constexpr int NSTAGE = 4;
  static constexpr int pa(int) { return 0; }
  static constexpr int pb(int) { return 0; }
};
struct KGrad13 : KindBase<2, 1, 2, 7u> {
  static constexpr int NSTAGE = 3;
  static constexpr int pa(int p) { return p; }
  static constexpr int pb(int) { return 0; }
};
struct KGrad2 : KindBase<1, 1, 1, 3u> {
  static constexpr int NSTAGE = 4;
  static constexpr int pa(int) { return 0; }
  static constexpr int pb(int) { return 0; }
};

// Newton-Schulz products: both operands K-contiguous, both row-contiguous, or
// only the second row-contiguous (B Y with Y read down its columns).
using KNsK = KOut;
using KNsMN = KGrad2;
struct KNsBY : KindBase<1, 1, 1, 2u> {
  static constexpr int NSTAGE = 4;
  static constexpr int pa(int) { return 0; }
  static constexpr int pb(int) { return 0; }
};

template <typename T, class K>
__device__ __forceinline__ void compute_ktile(const uint8_t* buf, f32x16_t (&acc)[K::NACC][2][2]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int arow = (w >> 1) * 64 + (lane & 31), brow = (w & 1) * 64 + (lane & 31);
  const int half = lane >> 5;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      u32x4_t af[K::NA][2], bf[K::NB][2];
#pragma unroll
      for (int o = 0; o < K::NA; ++o)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
          af[o][mi] = frag<T>(buf + o * kTileBytes, arow + mi * 32, 2 * s + half, K::is_mn(o));
#pragma unroll
      for (int o = 0; o < K::NB; ++o)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          bf[o][ni] = frag<T>(buf + (K::NA + o) * kTileBytes, brow + ni * 32, 2 * s + half,
                                      K::is_mn(K::NA + o));
#pragma unroll
      for (int p = 0; p < K::NACC; ++p)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
          for (int ni = 0; ni < 2; ++ni)
            if constexpr (__is_same(T, _Float16))
              acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
                  __builtin_bit_cast(f16x8_t, af[K::pa(p)][mi]),
                  __builtin_bit_cast(f16x8_t, bf[K::pb(p)][ni]), acc[p][mi][ni], 0, 0, 0);
            else
              acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  __builtin_bit_cast(bf16x8_t, af[K::pa(p)][mi]),
                  __builtin_bit_cast(bf16x8_t, bf[K::pb(p)][ni]), acc[p][mi][ni], 0, 0, 0);
    }
  } else {
    // fp32: lanes 0-31 hold K 0..7 of the tile, lanes 32-63 K 8..15; MFMA s
    // contracts K s (first half-wave) and K 8+s (second half-wave).
    float af[K::NA][2][8], bf[K::NB][2][8];
#pragma unroll
    for (int o = 0; o < K::NA; ++o)
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        // whole-vector bit casts: a bit cast of one vector element is not
        // reliable with this compiler (it reads element 0)
        const f32x4_t lo = __builtin_bit_cast(
            f32x4_t, frag<T>(buf + o * kTileBytes, arow + mi * 32, 2 * half, K::is_mn(o)));
        const f32x4_t hi = __builtin_bit_cast(
            f32x4_t, frag<T>(buf + o * kTileBytes, arow + mi * 32, 2 * half + 1, K::is_mn(o)));
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
        const f32x4_t lo =
            __builtin_bit_cast(f32x4_t, frag<T>(t, brow + ni * 32, 2 * half, K::is_mn(K::NA + o)));
        const f32x4_t hi =
            __builtin_bit_cast(f32x4_t, frag<T>(t, brow + ni * 32, 2 * half + 1, K::is_mn(K::NA + o)));
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
            acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                af[K::pa(p)][mi][s], bf[K::pb(p)][ni][s], acc[p][mi][ni], 0, 0, 0);
  }
}

// fp32 operands: register-staged double buffer (global -> VGPR -> LDS, with
// the in-register transposition of row-contiguous operands).
template <typename T, class K>
__device__ __forceinline__ void mainloop_regs(uint8_t* smem, const View (&ops)[K::NOPS], int64_t nk,
                                              f32x16_t (&acc)[K::NACC][2][2]) {
  constexpr int BK = Tr<T>::BK;
#pragma unroll
  for (int p = 0; p < K::NACC; ++p)
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[p][mi][ni][r] = 0.f;
  const int nkt = (int)((nk + BK - 1) / BK);
  if (nkt <= 0) return;

  u32x4_t st[K::NOPS][4];
  auto gload = [&](int64_t k0) {
#pragma unroll
    for (int o = 0; o < K::NOPS; ++o) {
      if constexpr (true) {
        if (K::is_mn(o)) {
          const int tt = threadIdx.x - 128 * K::mn_half(o);
          if (tt >= 0 && tt < 128) gload_mn<T>(st[o], ops[o], k0, tt);
        } else {
          gload_k<T>(st[o], ops[o], k0);
        }
      }
    }
  };
  auto sstore = [&](uint8_t* buf) {
#pragma unroll
    for (int o = 0; o < K::NOPS; ++o) {
      if (K::is_mn(o)) {
        const int tt = threadIdx.x - 128 * K::mn_half(o);
        if (tt >= 0 && tt < 128) sstore_mn<T>(buf + o * kTileBytes, st[o], tt);
      } else {
        sstore_k<T>(buf + o * kTileBytes, st[o]);
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
    compute_ktile<T, K>(cur, acc);
    if (more) sstore(smem + ((kt + 1) & 1) * K::NOPS * kTileBytes);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// 16-bit operands: direct global -> LDS DMA (global_load_lds_dwordx4) into a
// ring of K::NSTAGE stages, K::NSTAGE - 1 k-tiles in flight, no register
// staging. Row-contiguous operands keep their HBM layout in LDS (32 K rows x
// 256 bytes) and are read with ds_read_b64_tr_b16, which hands every lane
// four consecutive K of one row of the operand.

// A 16-byte page of zeros: out-of-range lanes load from it, so partial tiles
// arrive zero-padded in LDS.
__device__ __attribute__((aligned(64))) uint32_t g_zero_page[16];

// XOR swizzle of the 16-byte chunks of a row-contiguous tile (256-byte rows):
// the four K rows read by one 16-lane group of a transpose read land on
// distinct chunk positions.
__device__ __forceinline__ int swz_mn(int kr) { return (kr & 3) << 2; }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt_hi[15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_void_t;
typedef __attribute__((ext_vector_type(4))) short s16x4_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

__device__ __forceinline__ lds_void_t* to_lds(const void* p) {
  return (lds_void_t*)(p);
}

// Issue this wave's two 1 KiB DMA loads of one operand tile (512 chunks).
template <bool MN>
__device__ __forceinline__ void dma_tile(uint8_t* tile, const View& v, int64_t k0) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int base = w * 128 + i * 64;     // first 16-byte slot of this instruction
    const int p = base + lane;
    const uint8_t* src;
    if (!MN) {
      const int row = p >> 2;
      const int c = (p & 3) ^ (((row >> 1) ^ (row >> 3)) & 3);
      const int64_t k = k0 + c * 8;
      src = (row < v.nrows && k < v.nk) ? v.p + row * v.ld_b + k * 2
                                        : reinterpret_cast<const uint8_t*>(g_zero_page);
    } else {
      const int kr = p >> 4;
      const int c = (p & 15) ^ swz_mn(kr);
      const int64_t k = k0 + kr;
      src = (k < v.nk && c * 8 < v.nrows) ? v.p + k * v.ld_b + c * 16
                                          : reinterpret_cast<const uint8_t*>(g_zero_page);
    }
    __builtin_amdgcn_global_load_lds((gbl_void_t*)src, to_lds(tile + base * 16), 16, 0, 0);
  }
}

// MFMA fragment (8 consecutive K of row rb + lane%32, K block 8*(lane/32) of
// substep s) from a row-contiguous tile, by two transpose reads. Issued as
// inline asm so the compiler does not drain the in-flight DMA before it (it
// cannot tell which stage the read touches); the result is not ready until a
// lgkm_ready() on it.
__device__ __forceinline__ u32x4_t frag_tr(const uint8_t* tile, int rb, int s) {
  const int lane = threadIdx.x & 63, g = lane >> 4, sl = lane & 15;
  const int mn = rb + 16 * (g & 1) + 4 * (sl & 3);
  const int c = mn >> 3, hb = (mn >> 2) & 1;
  const uint32_t base = (uint32_t)(uintptr_t)to_lds(tile);
  u32x2_t lo, hi;
  {
    const int kr = 16 * s + 8 * (g >> 1) + (sl >> 2);
    const uint32_t a = base + kr * 256 + ((c ^ swz_mn(kr)) << 4) + (hb << 3);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a));
  }
  {
    const int kr = 16 * s + 8 * (g >> 1) + 4 + (sl >> 2);
    const uint32_t a = base + kr * 256 + ((c ^ swz_mn(kr)) << 4) + (hb << 3);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(hi) : "v"(a));
  }
  return u32x4_t{lo[0], lo[1], hi[0], hi[1]};
}

// Waits for outstanding LDS reads and makes `x` depend on the wait, so no use
// of a transpose-read result is scheduled before its data has arrived.
__device__ __forceinline__ void lgkm_ready(u32x4_t& x) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(x));
}

template <typename T, class K>
__device__ __forceinline__ void compute_ktile16(const uint8_t* buf, f32x16_t (&acc)[K::NACC][2][2]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ab = (w >> 1) * 64, bb = (w & 1) * 64;
  const int arow = ab + (lane & 31), brow = bb + (lane & 31);
  const int half = lane >> 5;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    u32x4_t af[K::NA][2], bf[K::NB][2];
#pragma unroll
    for (int o = 0; o < K::NA; ++o)
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        af[o][mi] = K::is_mn(o) ? frag_tr(buf + o * kTileBytes, ab + mi * 32, s)
                                : frag<T>(buf + o * kTileBytes, arow + mi * 32, 2 * s + half, false);
#pragma unroll
    for (int o = 0; o < K::NB; ++o)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bf[o][ni] = K::is_mn(K::NA + o)
                        ? frag_tr(buf + (K::NA + o) * kTileBytes, bb + ni * 32, s)
                        : frag<T>(buf + (K::NA + o) * kTileBytes, brow + ni * 32, 2 * s + half, false);
    if constexpr (K::MN != 0u) {
#pragma unroll
      for (int o = 0; o < K::NA; ++o)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
          if (K::is_mn(o)) lgkm_ready(af[o][mi]);
#pragma unroll
      for (int o = 0; o < K::NB; ++o)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          if (K::is_mn(K::NA + o)) lgkm_ready(bf[o][ni]);
    }
#pragma unroll
    for (int p = 0; p < K::NACC; ++p)
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          if constexpr (__is_same(T, _Float16))
            acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
                __builtin_bit_cast(f16x8_t, af[K::pa(p)][mi]),
                __builtin_bit_cast(f16x8_t, bf[K::pb(p)][ni]), acc[p][mi][ni], 0, 0, 0);
          else
            acc[p][mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, af[K::pa(p)][mi]),
                __builtin_bit_cast(bf16x8_t, bf[K::pb(p)][ni]), acc[p][mi][ni], 0, 0, 0);
        }
  }
}

template <typename T, class K>
__device__ __forceinline__ void mainloop_dma(uint8_t* smem, const View (&ops)[K::NOPS], int64_t nk,
                                             f32x16_t (&acc)[K::NACC][2][2]) {
  constexpr int BK = 32, NS = K::NSTAGE, STAGE = K::NOPS * kTileBytes;
  constexpr int L = 2 * K::NOPS;   // DMA instructions per wave per k-tile
#pragma unroll
  for (int p = 0; p < K::NACC; ++p)
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[p][mi][ni][r] = 0.f;
  const int nkt = (int)((nk + BK - 1) / BK);
  if (nkt <= 0) return;
  auto issue = [&](int kt) {
    uint8_t* st = smem + (kt % NS) * STAGE;
#pragma unroll
    for (int o = 0; o < K::NOPS; ++o) {
      if (K::is_mn(o)) dma_tile<true>(st + o * kTileBytes, ops[o], (int64_t)kt * BK);
      else dma_tile<false>(st + o * kTileBytes, ops[o], (int64_t)kt * BK);
    }
  };
#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < nkt) issue(t);
  for (int kt = 0; kt < nkt; ++kt) {
    // this wave's loads of tile kt are done once at most the later tiles' are pending
    if (kt + NS - 2 < nkt) wait_vmcnt<L * (NS - 2)>();
    else wait_vmcnt<0>();
    // every wave's tile kt is in LDS and tile kt-1's stage is free; a bare
    // barrier (a fenced one would drain all DMA still in flight)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (kt + NS - 1 < nkt) issue(kt + NS - 1);
    compute_ktile16<T, K>(smem + (kt % NS) * STAGE, acc);
  }
  __syncthreads();     // the caller may reuse LDS after the loop
}

template <typename T, class K>
__device__ __forceinline__ void mainloop(uint8_t* smem, const View (&ops)[K::NOPS], int64_t nk,
                                         f32x16_t (&acc)[K::NACC][2][2]) {
  if constexpr (sizeof(T) == 2) mainloop_dma<T, K>(smem, ops, nk, acc);
  else mainloop_regs<T, K>(smem, ops, nk, acc);
}

template <class K>
constexpr int smem_bytes() {
  const int dma = K::NSTAGE * K::NOPS * kTileBytes, regs = 2 * K::NOPS * kTileBytes;
  return dma > regs ? dma : regs;
}
constexpr int cmax(int a, int b) { return a > b ? a : b; }

// Epilogue coordinates of accumulator register r of block (mi, ni).
__device__ __forceinline__ int acc_row(int mi, int r) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  return (w >> 1) * 64 + mi * 32 + ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3);
}
__device__ __forceinline__ int acc_col(int ni) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  return (w & 1) * 64 + ni * 32 + (lane & 31);
}

template <typename T>
__device__ __forceinline__ void st_elem(void* base, int64_t idx, float v) {
  reinterpret_cast<T*>(base)[idx] = (T)v;
}

__device__ __forceinline__ float sigmoidf_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

__device__ __forceinline__ View view_k(const Operand& op, int inst, int64_t row0, int64_t k0,
                                       int64_t nrows, int64_t nk, int esz) {
  const int64_t off = inst * op.inst_stride + row0 * op.ld + k0;
  return View{reinterpret_cast<const uint8_t*>(op.base) + off * esz, op.ld * esz, nrows, nk};
}
__device__ __forceinline__ View view_mn(const Operand& op, int inst, int64_t row0, int64_t k0,
                                        int64_t nrows, int64_t nk, int esz) {
  const int64_t off = inst * op.inst_stride + k0 * op.ld + row0;
  return View{reinterpret_cast<const uint8_t*>(op.base) + off * esz, op.ld * esz, nrows, nk};
}

// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_fwd(const FwdArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[cmax(smem_bytes<KApply>(), smem_bytes<KUpdate>())];
  constexpr int esz = sizeof(T);
  int bid = xcd_remap(blockIdx.x, args.total_blocks);
  const bool first = bid < args.seg[0].nblocks;
  const FwdSeg& sg = first ? args.seg[0] : args.seg[1];
  if (!first) bid -= args.seg[0].nblocks;
  const int per = sg.tiles_m * sg.tiles_n;
  const int inst = bid / per;
  const int rr = bid - inst * per;
  const int64_t i0 = (int64_t)(rr / sg.tiles_n) * kTile;   // token tile
  const int64_t j0 = (int64_t)(rr % sg.tiles_n) * kTile;   // hidden tile
  const int d = args.d, h = args.h;
  const int64_t mrows = sg.rows - i0, ncols = h - j0;

  if (sg.kind == FWD_APPLY) {
    const View ops[3] = {view_k(sg.a0, inst, i0, 0, mrows, d, esz),
                         view_k(args.w1, inst, j0, 0, ncols, d, esz),
                         view_k(args.w3, inst, j0, 0, ncols, d, esz)};
    f32x16_t acc[2][2][2];
    mainloop<T, KApply>(smem, ops, d, acc);
    void* out = reinterpret_cast<uint8_t*>(sg.out0) + (inst * sg.out_inst) * esz;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = acc_col(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row(mi, r);
          if (i < mrows && j < ncols) {
            const float z1 = acc[0][mi][ni][r], z3 = acc[1][mi][ni][r];
            st_elem<T>(out, (i0 + i) * h + j0 + j, z1 * sigmoidf_fast(z1) * z3);
          }
        }
      }
  } else {
    const View ops[5] = {view_k(sg.a0, inst, i0, 0, mrows, d, esz),
                         view_k(sg.a1, inst, i0, 0, mrows, d, esz),
                         view_k(args.w1, inst, j0, 0, ncols, d, esz),
                         view_k(args.w3, inst, j0, 0, ncols, d, esz),
                         view_mn(args.w2, inst, j0, 0, ncols, d, esz)};
    f32x16_t acc[3][2][2];
    mainloop<T, KUpdate>(smem, ops, d, acc);
    const int64_t ob = inst * sg.out_inst;
    const float* eta = sg.eta + inst * sg.eta_inst + i0;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
      float e[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = acc_row(mi, r);
        e[r] = i < mrows ? eta[i] : 0.f;
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = acc_col(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row(mi, r);
          if (i < mrows && j < ncols) {
            const float z1 = acc[0][mi][ni][r], z3 = acc[1][mi][ni][r], dh = acc[2][mi][ni][r];
            const float s = sigmoidf_fast(z1);
            const float a = z1 * s;                       // SiLU(z1)
            const float ed = e[r] * dh;                   // eta_i * (W2^T v_i)_j
            const int64_t idx = ob + (i0 + i) * h + j0 + j;
            st_elem<T>(sg.out1, idx, e[r] * a * z3);                          // eta * hidden
            st_elem<T>(sg.out2, idx, ed * z3 * s * (1.0f + z1 * (1.0f - s))); // eta * dz1
            st_elem<T>(sg.out3, idx, ed * a);                                 // eta * dz3
          }
        }
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_bwd(const BwdArgs args) {
  __shared__ __attribute__((aligned(16)))
  uint8_t smem[cmax(smem_bytes<KOut>(), cmax(smem_bytes<KGrad13>(), smem_bytes<KGrad2>()))];
  constexpr int esz = sizeof(T);
  int bid = xcd_remap(blockIdx.x, args.total_blocks);
  int si = 0;
  if (bid >= args.seg[0].nblocks) {
    bid -= args.seg[0].nblocks;
    si = 1;
    if (bid >= args.seg[1].nblocks) {
      bid -= args.seg[1].nblocks;
      si = 2;
    }
  }
  const BwdSeg& sg = si == 0 ? args.seg[0] : (si == 1 ? args.seg[1] : args.seg[2]);
  const int d = args.d, h = args.h;
  const int per = sg.tiles_m * sg.tiles_n;
  const int per_inst = per * sg.nsplit;
  const int inst = bid / per_inst;
  int rr = bid - inst * per_inst;
  const int split = rr / per;
  rr -= split * per;
  const int64_t r0 = (int64_t)(rr / sg.tiles_n) * kTile;
  const int64_t c0 = (int64_t)(rr % sg.tiles_n) * kTile;

  if (sg.kind == BWD_OUT) {
    // O[i, m] = sum_j hidden[i, j] W2[m, j]
    const int64_t mrows = sg.rows - r0, ncols = d - c0;
    const View ops[2] = {view_k(sg.a0, inst, r0, 0, mrows, h, esz),
                         view_k(sg.b0, inst, c0, 0, ncols, h, esz)};
    f32x16_t acc[1][2][2];
    mainloop<T, KOut>(smem, ops, h, acc);
    const int64_t ob = inst * sg.out_inst;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = acc_col(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row(mi, r);
          if (i < mrows && j < ncols) st_elem<T>(sg.out, ob + (r0 + i) * d + c0 + j, acc[0][mi][ni][r]);
        }
      }
    return;
  }

  const int64_t kb = (int64_t)split * sg.split_len;
  int64_t klen = sg.rows - kb;
  if (klen > sg.split_len) klen = sg.split_len;
  if (klen < 0) klen = 0;
  float* part = reinterpret_cast<float*>(sg.out) + split * sg.out_split + inst * sg.out_inst;
  const int64_t dh = (int64_t)d * h;
  if (sg.kind == BWD_GRAD13) {
    // P1[j, m] = sum_i (eta dz1)[i, j] K[i, m];  P3 likewise with eta dz3
    const int64_t mrows = h - r0, ncols = d - c0;
    const View ops[3] = {view_mn(sg.a0, inst, r0, kb, mrows, klen, esz),
                         view_mn(sg.a1, inst, r0, kb, mrows, klen, esz),
                         view_mn(sg.b0, inst, c0, kb, ncols, klen, esz)};
    f32x16_t acc[2][2][2];
    mainloop<T, KGrad13>(smem, ops, klen, acc);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = acc_col(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row(mi, r);
          if (i < mrows && j < ncols) {
            const int64_t idx = (r0 + i) * d + c0 + j;
            part[idx] = acc[0][mi][ni][r];
            part[2 * dh + idx] = acc[1][mi][ni][r];
          }
        }
      }
  } else {
    // P2[m, j] = sum_i V[i, m] (eta hidden)[i, j]
    const int64_t mrows = d - r0, ncols = h - c0;
    const View ops[2] = {view_mn(sg.a0, inst, r0, kb, mrows, klen, esz),
                         view_mn(sg.b0, inst, c0, kb, ncols, klen, esz)};
    f32x16_t acc[1][2][2];
    mainloop<T, KGrad2>(smem, ops, klen, acc);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = acc_col(ni);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = acc_row(mi, r);
          if (i < mrows && j < ncols) part[dh + (r0 + i) * h + c0 + j] = acc[0][mi][ni][r];
        }
      }
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// One wave per row of W1 (length d), W2 (length h) or W3 (length d):
//   U = W + sum_split P  (P = -g, the negated gradient or its Newton-Schulz image)
//   W <- U * ||W_row|| / ||U_row||       (§3.2 weight normalisation; Alg. 1)
template <typename T>
__global__ __launch_bounds__(kThreads) void k_update(const UpdArgs a) {
  const int wave = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wave >= a.rows_total) return;
  const int rows_inst = 2 * a.h + a.d;
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
  const int64_t dh = (int64_t)a.d * a.h;
  const int64_t off = inst * dh + (int64_t)r * L;
  float* W = a.W[mat] + off;
  const float* P = a.step + inst * 3 * dh + mat * dh + (int64_t)r * L;
  constexpr int kPer = kMaxDim / 64;
  float u[kPer];
  float sw = 0.f, su = 0.f;
#pragma unroll
  for (int t = 0; t < kPer; ++t) {
    const int c = lane + 64 * t;
    u[t] = 0.f;
    if (c < L) {
      const float w = W[c];
      float p = 0.f;
      for (int s = 0; s < a.nsplit; ++s) p += P[s * a.step_split + c];
      const float x = w + p;
      u[t] = x;
      sw += w * w;
      su += x * x;
    }
  }
  sw = wave_sum(sw);
  su = wave_sum(su);
  const float scale = sqrtf(sw) / sqrtf(su);
  void* wb = a.Wb[mat];
#pragma unroll
  for (int t = 0; t < kPer; ++t) {
    const int c = lane + 64 * t;
    if (c < L) {
      const float x = u[t] * scale;
      W[c] = x;
      if constexpr (sizeof(T) == 2) reinterpret_cast<__bf16*>(wb)[off + c] = (__bf16)x;
    }
  }
}

__global__ __launch_bounds__(kThreads) void k_prep(const float* w1, const float* w2, const float* w3,
                                                   __bf16* b1, __bf16* b2, __bf16* b3, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) {
    b1[i] = (__bf16)w1[i];
    b2[i] = (__bf16)w2[i];
    b3[i] = (__bf16)w3[i];
  }
}

// One Newton-Schulz product over every matrix of the chunk (see NsKind).
template <typename T>
__global__ __launch_bounds__(kThreads) void k_ns(const NsArgs args) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[cmax(smem_bytes<KNsK>(), smem_bytes<KNsBY>())];
  constexpr int esz = sizeof(T);
  int bid = xcd_remap(blockIdx.x, args.total_blocks);
  const bool first = bid < args.seg[0].nblocks;
  const NsSeg& sg = first ? args.seg[0] : args.seg[1];
  if (!first) bid -= args.seg[0].nblocks;
  const int per = sg.tiles_m * sg.tiles_n;
  const int q = bid / per;
  const int rr = bid - q * per;
  const int64_t i0 = (int64_t)(rr / sg.tiles_n) * kTile, j0 = (int64_t)(rr % sg.tiles_n) * kTile;
  const int64_t slot = (int64_t)(q / sg.group) * 3 + sg.slot_off[q % sg.group];
  const int m = args.m, ldy = sg.ldy;
  const int64_t mrows = sg.M - i0, ncols = sg.N - j0;
  float* Y32 = args.Y32 + slot * args.ystride;
  const uint8_t* Yin = reinterpret_cast<const uint8_t*>(args.Yin) + slot * args.ystride * esz;
  void* Yout = reinterpret_cast<uint8_t*>(args.Yout) + slot * args.ystride * esz;
  float* A32 = args.A32 + slot * args.astride;
  const uint8_t* Ab = reinterpret_cast<const uint8_t*>(args.Ab) + slot * args.astride * esz;
  void* Abw = reinterpret_cast<uint8_t*>(args.Ab) + slot * args.astride * esz;
  const uint8_t* Bb = reinterpret_cast<const uint8_t*>(args.Bb) + slot * args.astride * esz;
  void* Bbw = reinterpret_cast<uint8_t*>(args.Bb) + slot * args.astride * esz;
  f32x16_t acc[1][2][2];
  const int kind = sg.kind;
  if (kind == NS_GRAM_K) {          // A = Y Y^T
    const View ops[2] = {View{Yin + i0 * ldy * esz, (int64_t)ldy * esz, mrows, sg.K},
                         View{Yin + j0 * ldy * esz, (int64_t)ldy * esz, ncols, sg.K}};
    mainloop<T, KNsK>(smem, ops, sg.K, acc);
  } else if (kind == NS_GRAM_MN) {  // A = Y^T Y
    const View ops[2] = {View{Yin + i0 * esz, (int64_t)ldy * esz, mrows, sg.K},
                         View{Yin + j0 * esz, (int64_t)ldy * esz, ncols, sg.K}};
    mainloop<T, KNsMN>(smem, ops, sg.K, acc);
  } else if (kind == NS_POLY) {     // A A (A symmetric, so A A^T)
    const View ops[2] = {View{Ab + i0 * m * esz, (int64_t)m * esz, mrows, sg.K},
                         View{Ab + j0 * m * esz, (int64_t)m * esz, ncols, sg.K}};
    mainloop<T, KNsK>(smem, ops, sg.K, acc);
  } else if (kind == NS_UPD_BY) {   // B Y
    const View ops[2] = {View{Bb + i0 * m * esz, (int64_t)m * esz, mrows, sg.K},
                         View{Yin + j0 * esz, (int64_t)ldy * esz, ncols, sg.K}};
    mainloop<T, KNsBY>(smem, ops, sg.K, acc);
  } else {                          // Y B (B symmetric)
    const View ops[2] = {View{Yin + i0 * ldy * esz, (int64_t)ldy * esz, mrows, sg.K},
                         View{Bb + j0 * m * esz, (int64_t)m * esz, ncols, sg.K}};
    mainloop<T, KNsK>(smem, ops, sg.K, acc);
  }
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int j = acc_col(ni);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = acc_row(mi, r);
        if (i < mrows && j < ncols) {
          const float v = acc[0][mi][ni][r];
          if (kind == NS_GRAM_K || kind == NS_GRAM_MN) {
            const int64_t idx = (i0 + i) * m + j0 + j;
            A32[idx] = v;
            st_elem<T>(Abw, idx, v);
          } else if (kind == NS_POLY) {
            const int64_t idx = (i0 + i) * m + j0 + j;
            st_elem<T>(Bbw, idx, args.cb * A32[idx] + args.cc * v);
          } else {
            const int64_t idx = (i0 + i) * ldy + j0 + j;
            const float y = args.ca * Y32[idx] + v;
            Y32[idx] = y;
            st_elem<T>(Yout, idx, y);
          }
        }
      }
    }
}

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) t += red[i];
  __syncthreads();
  return t;
}

// Sum the split-K partials of every gradient and the per-block sums of squares.
__global__ __launch_bounds__(kThreads) void k_ns_prep(const NsPrepArgs a) {
  __shared__ float red[kThreads / 64];
  const int slot = blockIdx.x / a.blocks_per_slot;
  const int blk = blockIdx.x - slot * a.blocks_per_slot;
  const int64_t base = (int64_t)slot * a.dh;
  float ss = 0.f;
  for (int e = threadIdx.x; e < kNsBlockElems; e += kThreads) {
    const int64_t idx = (int64_t)blk * kNsBlockElems + e;
    if (idx < a.dh) {
      float g = 0.f;
      for (int s = 0; s < a.nsplit; ++s) g += a.part[s * a.part_split + base + idx];
      a.Y32[base + idx] = g;
      ss += g * g;
    }
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) a.sumsq[(int64_t)slot * a.blocks_per_slot + blk] = ss;
}

// X0 = G / (||G||_F + eps), fp32 iterate and operand copy.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_ns_scale(const NsPrepArgs a, void* yb, float eps) {
  __shared__ float red[kThreads / 64];
  const int slot = blockIdx.x / a.blocks_per_slot;
  const int blk = blockIdx.x - slot * a.blocks_per_slot;
  const int64_t base = (int64_t)slot * a.dh;
  float t = 0.f;
  for (int b = threadIdx.x; b < a.blocks_per_slot; b += kThreads)
    t += a.sumsq[(int64_t)slot * a.blocks_per_slot + b];
  t = block_sum(t, red);
  const float inv = 1.0f / (sqrtf(t) + eps);
  for (int e = threadIdx.x; e < kNsBlockElems; e += kThreads) {
    const int64_t idx = (int64_t)blk * kNsBlockElems + e;
    if (idx < a.dh) {
      const float y = a.Y32[base + idx] * inv;
      a.Y32[base + idx] = y;
      st_elem<T>(yb, base + idx, y);
    }
  }
}

}  // namespace

hipError_t launch_ns(const NsArgs& a, bool fp16, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  if (fp16) k_ns<_Float16><<<a.total_blocks, kThreads, 0, s>>>(a);
  else k_ns<float><<<a.total_blocks, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_ns_prep(const NsPrepArgs& a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.nslots * a.blocks_per_slot;
  if (blocks <= 0) return hipSuccess;
  k_ns_prep<<<(unsigned)blocks, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_ns_scale(const NsPrepArgs& a, void* Yb, bool fp16, float eps, hipStream_t s) {
  const int64_t blocks = (int64_t)a.nslots * a.blocks_per_slot;
  if (blocks <= 0) return hipSuccess;
  if (fp16) k_ns_scale<_Float16><<<(unsigned)blocks, kThreads, 0, s>>>(a, Yb, eps);
  else k_ns_scale<float><<<(unsigned)blocks, kThreads, 0, s>>>(a, Yb, eps);
  return hipGetLastError();
}

hipError_t launch_fwd(const FwdArgs& a, bool io_bf16, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  if (io_bf16) k_fwd<__bf16><<<a.total_blocks, kThreads, 0, s>>>(a);
  else k_fwd<float><<<a.total_blocks, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdArgs& a, bool io_bf16, hipStream_t s) {
  if (a.total_blocks <= 0) return hipSuccess;
  if (io_bf16) k_bwd<__bf16><<<a.total_blocks, kThreads, 0, s>>>(a);
  else k_bwd<float><<<a.total_blocks, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_update(const UpdArgs& a, bool io_bf16, hipStream_t s) {
  const int waves_per_block = kThreads / 64;
  const int blocks = (a.rows_total + waves_per_block - 1) / waves_per_block;
  if (blocks <= 0) return hipSuccess;
  if (io_bf16) k_update<__bf16><<<blocks, kThreads, 0, s>>>(a);
  else k_update<float><<<blocks, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_prep(const float* const W[3], void* const Wb[3], int BH, int d, int h, hipStream_t s) {
  const int64_t n = (int64_t)BH * d * h;
  const int64_t blocks = (n + kThreads - 1) / kThreads;
  if (blocks <= 0) return hipSuccess;
  k_prep<<<(unsigned)blocks, kThreads, 0, s>>>(W[0], W[1], W[2], reinterpret_cast<__bf16*>(Wb[0]),
                                              reinterpret_cast<__bf16*>(Wb[1]),
                                              reinterpret_cast<__bf16*>(Wb[2]), n);
  return hipGetLastError();
}

}  // namespace lact
