// The steps of the LaCT layer on either side of the fast-weight path (Alg. 1,
// layer): the prologue that turns the q/k/v projections and the raw rates into
// the path's inputs, and the per-head RMSNorm of its output. Both are one pass
// over HBM: every input byte is read once and every output byte written once.
//
// A "group" of G lanes (G a power of two, G <= 64) owns (token, head) vectors
// of hd elements; each lane moves 16 bytes per access, NV accesses per vector,
// and the group's sum of squares is a shuffle reduction within it.
#include "lact_internal.h"

namespace lact {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_io;

template <typename T> struct Io;
template <> struct Io<__bf16> {
  static constexpr int EPV = 8;   // elements per 16-byte access
  __device__ static void load(const void* p, float (&x)[8]) {
    const u32x4_io u = *reinterpret_cast<const u32x4_io*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(u[i] << 16);
      x[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
    }
  }
  __device__ static void store(void* p, const float (&x)[8]) {
    typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
    bf16x8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i) b[i] = (__bf16)x[i];
    *reinterpret_cast<bf16x8*>(p) = b;
  }
};
template <> struct Io<float> {
  static constexpr int EPV = 4;
  // n (4 or 8) consecutive floats
  __device__ static void load8(const float* p, float (&x)[8], int n) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
    if (n > 4) {
      const float4 w = *reinterpret_cast<const float4*>(p + 4);
      x[4] = w.x; x[5] = w.y; x[6] = w.z; x[7] = w.w;
    }
  }
  __device__ static void load(const void* p, float (&x)[8]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  __device__ static void store(void* p, const float (&x)[8]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
};

// (token t, head hh) of vector g = t * H + hh, and token t = b * L + l. The
// divisions run in 32 bits when every index fits (IX = uint32_t): a 64-bit
// division per vector costs more ALU time than the vector's memory traffic.
template <typename IX>
__device__ __forceinline__ void split_g(int64_t g, int H, int64_t L, int& hh, int64_t& t, int64_t& b, int64_t& l) {
  const IX gi = (IX)g, hi = (IX)H, Li = (IX)L;
  const IX ti = gi / hi;
  hh = (int)(gi - ti * hi);
  const IX bi = ti / Li;
  l = (int64_t)(ti - bi * Li);
  t = (int64_t)ti;
  b = (int64_t)bi;
}

__device__ __forceinline__ float group_sum(float v, int G) {
  for (int off = G >> 1; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float sigmoid_acc(float x) { return 1.0f / (1.0f + expf(-x)); }

// SiLU with the hardware exp2 and reciprocal (about 1 ulp each): the prologue
// applies it to every input element, so the IEEE exp and divide would make the
// kernel bound by ALU work instead of HBM.
__device__ __forceinline__ float silu_fast(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -1.4426950408889634f));
}

// log(1 + e^x) without overflow: max(x, 0) + log1p(e^-|x|)
__device__ __forceinline__ float softplus_acc(float x) { return fmaxf(x, 0.0f) + log1pf(expf(-fabsf(x))); }

// Each group takes U consecutive (token, head) vectors per iteration and issues
// every load of all of them (q, k and v) before it computes anything. Measured
// on MI355X at the LM shape: U = 1 (5.1 TB/s prologue, 5.4 TB/s norm) beats
// U = 2..8 (down to 3.6 and 3.9 TB/s): the registers of more vectors per wave
// cost more waves in flight than they add loads.
template <typename T, int NV, int U, typename IX>
__global__ __launch_bounds__(256) void k_prologue(const PrologueArgs a) {
  constexpr int EPV = Io<T>::EPV;
  const int G = a.group;
  const int lane_g = threadIdx.x & (G - 1);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H, nsuper = (ngroups + U - 1) / U;
  const int64_t gstride = (int64_t)gridDim.x * (256 / G);
  const int nvec = a.hd / EPV;   // 16-byte accesses per vector
  for (int64_t sg = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G; sg < nsuper; sg += gstride) {
    float x[U][3][NV][8];
    int64_t tt[U], ll[U], in[U];
    bool ok[U], kv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t g = sg * U + u;
      ok[u] = g < ngroups;
      int hh;
      int64_t b;
      split_g<IX>(g, a.H, a.L, hh, tt[u], b, ll[u]);
      in[u] = b * a.H + hh;
      kv[u] = ok[u] && ll[u] < a.n_kv;  // k, v and rates exist for key tokens only
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        if (!(p == 0 ? ok[u] : kv[u])) continue;
        const T* src = reinterpret_cast<const T*>(a.qkv) + ((tt[u] * 3 + p) * a.H + hh) * a.hd;
#pragma unroll
        for (int j = 0; j < NV; ++j)
          if (lane_g + j * G < nvec) Io<T>::load(src + (lane_g + j * G) * EPV, x[u][p][j]);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        float ss = 0.0f;
        const bool live = p == 0 ? ok[u] : kv[u];
#pragma unroll
        for (int j = 0; j < NV; ++j)
          if (live && lane_g + j * G < nvec)
#pragma unroll
            for (int e = 0; e < EPV; ++e) {
              x[u][p][j][e] = silu_fast(x[u][p][j][e]);
              ss += x[u][p][j][e] * x[u][p][j][e];
            }
        float scale = 1.0f;
        if (p < 2) {                    // q / ||q||, k / ||k||; a zero vector stays zero
          ss = group_sum(ss, G);        // the whole group shares `live`
          scale = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
        }
        if (!live) continue;
        T* dst = reinterpret_cast<T*>(p == 0 ? a.q : (p == 1 ? a.k : a.v)) +
                 (in[u] * (p == 0 ? a.L : a.n_kv) + ll[u]) * a.hd;
#pragma unroll
        for (int j = 0; j < NV; ++j)
          if (lane_g + j * G < nvec) {
#pragma unroll
            for (int e = 0; e < EPV; ++e) x[u][p][j][e] *= scale;
            Io<T>::store(dst + (lane_g + j * G) * EPV, x[u][p][j]);
          }
      }
      if (kv[u]) {                      // learning rates: softplus(raw + bias)
        const int hh = (int)(in[u] - (in[u] / a.H) * a.H);
        for (int r = lane_g; r < a.R; r += G)
          a.eta[(in[u] * a.n_kv + ll[u]) * a.R + r] =
              softplus_acc(a.lr_raw[(tt[u] * a.H + hh) * a.R + r] + a.lr_bias);
        if (a.beta && lane_g == 0) a.beta[in[u] * a.n_kv + ll[u]] = sigmoid_acc(a.beta_raw[tt[u] * a.H + hh]);
      }
    }
  }
}

template <typename T, int NV, int U, typename IX>
__global__ __launch_bounds__(256) void k_rmsnorm_out(const RmsArgs a) {
  constexpr int EPV = Io<T>::EPV;
  const int G = a.group;
  const int lane_g = threadIdx.x & (G - 1);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H, nsuper = (ngroups + U - 1) / U;
  const int64_t gstride = (int64_t)gridDim.x * (256 / G);
  const int nvec = a.hd / EPV;
  for (int64_t sg = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G; sg < nsuper; sg += gstride) {
    // output order (b, l, h): consecutive vectors of a group are consecutive in y
    float x[U][NV][8], wv[U][NV][8];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t g = sg * U + u;
      ok[u] = g < ngroups;
      if (!ok[u]) continue;
      int hh;
      int64_t t, b, l;
      split_g<IX>(g, a.H, a.L, hh, t, b, l);
      const T* src = reinterpret_cast<const T*>(a.o) + ((b * a.H + hh) * a.L + l) * a.hd;
#pragma unroll
      for (int j = 0; j < NV; ++j)
        if (lane_g + j * G < nvec) {
          Io<T>::load(src + (lane_g + j * G) * EPV, x[u][j]);
          if (a.weight) Io<float>::load8(a.weight + (int64_t)hh * a.hd + (lane_g + j * G) * EPV, wv[u][j], EPV);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float ss = 0.0f;
#pragma unroll
      for (int j = 0; j < NV; ++j)
        if (ok[u] && lane_g + j * G < nvec)
#pragma unroll
          for (int e = 0; e < EPV; ++e) ss += x[u][j][e] * x[u][j][e];
      ss = group_sum(ss, G);
      if (!ok[u]) continue;
      const int64_t g = sg * U + u;
      const float inv = 1.0f / sqrtf(ss / (float)a.hd + a.eps);
      T* dst = reinterpret_cast<T*>(a.y) + g * a.hd;     // y[b, l, h] is vector g
#pragma unroll
      for (int j = 0; j < NV; ++j)
        if (lane_g + j * G < nvec) {
#pragma unroll
          for (int e = 0; e < EPV; ++e) x[u][j][e] *= a.weight ? inv * wv[u][j][e] : inv;
          Io<T>::store(dst + (lane_g + j * G) * EPV, x[u][j]);
        }
    }
  }
}

// Group size and accesses per lane for hd elements of esz bytes.
void io_shape(int hd, int esz, int& group, int& nv) {
  const int nvec = hd * esz / 16;
  group = 1;
  while (group < nvec && group < 64) group <<= 1;
  nv = (nvec + group - 1) / group;
}

int64_t io_blocks(int64_t nsuper, int group) {
  const int64_t need = (nsuper * group + 255) / 256;
  return need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20);
}

// vectors per group and iteration (see k_prologue)
template <int NV> constexpr int prologue_u() { return 1; }
template <int NV> constexpr int rms_u() { return 1; }

template <template <typename, int> class KER, typename T, typename A>
hipError_t launch_nv(const A& a, int nv, hipStream_t s) {
  switch (nv) {
    case 1: KER<T, 1>::launch(a, s); break;
    case 2: KER<T, 2>::launch(a, s); break;
    case 4: KER<T, 4>::launch(a, s); break;
    case 8: KER<T, 8>::launch(a, s); break;
    default: KER<T, 16>::launch(a, s); break;
  }
  return hipGetLastError();
}

template <typename T, int NV> struct PrologueK {
  static void launch(const PrologueArgs& a, hipStream_t s) {
    constexpr int U = prologue_u<NV>();
    const int64_t nsuper = ((int64_t)a.B * a.L * a.H + U - 1) / U;
    const unsigned blocks = (unsigned)io_blocks(nsuper, a.group);
    if ((int64_t)a.B * a.L * a.H < ((int64_t)1 << 31)) k_prologue<T, NV, U, uint32_t><<<blocks, 256, 0, s>>>(a);
    else k_prologue<T, NV, U, uint64_t><<<blocks, 256, 0, s>>>(a);
  }
};
template <typename T, int NV> struct RmsK {
  static void launch(const RmsArgs& a, hipStream_t s) {
    constexpr int U = rms_u<NV>();
    const int64_t nsuper = ((int64_t)a.B * a.L * a.H + U - 1) / U;
    const unsigned blocks = (unsigned)io_blocks(nsuper, a.group);
    if ((int64_t)a.B * a.L * a.H < ((int64_t)1 << 31)) k_rmsnorm_out<T, NV, U, uint32_t><<<blocks, 256, 0, s>>>(a);
    else k_rmsnorm_out<T, NV, U, uint64_t><<<blocks, 256, 0, s>>>(a);
  }
};

// hd <= 4096: at most 1024 accesses of 16 bytes per vector, 16 per lane
int round_nv(int nv) { return nv <= 1 ? 1 : nv <= 2 ? 2 : nv <= 4 ? 4 : nv <= 8 ? 8 : 16; }

}  // namespace

hipError_t launch_prologue(PrologueArgs a, bool io_bf16, hipStream_t s) {
  int nv;
  io_shape(a.hd, io_bf16 ? 2 : 4, a.group, nv);
  if ((int64_t)a.B * a.L * a.H <= 0) return hipSuccess;
  nv = round_nv(nv);
  return io_bf16 ? launch_nv<PrologueK, __bf16>(a, nv, s) : launch_nv<PrologueK, float>(a, nv, s);
}

hipError_t launch_rmsnorm_out(RmsArgs a, bool io_bf16, hipStream_t s) {
  int nv;
  io_shape(a.hd, io_bf16 ? 2 : 4, a.group, nv);
  if ((int64_t)a.B * a.L * a.H <= 0) return hipSuccess;
  nv = round_nv(nv);
  return io_bf16 ? launch_nv<RmsK, __bf16>(a, nv, s) : launch_nv<RmsK, float>(a, nv, s);
}

}  // namespace lact
