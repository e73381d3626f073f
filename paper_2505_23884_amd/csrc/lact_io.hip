// The steps of the LaCT layer on either side of the fast-weight path (Alg. 1,
// layer): the prologue that turns the q/k/v projections and the raw rates into
// the path's inputs, and the per-head RMSNorm of its output. Both are one pass
// over HBM: every input byte is read once and every output byte written once.
//
// A "group" of G lanes (G a power of two, G <= 64) owns one (token, head)
// vector of hd elements; each lane moves 16 bytes per access, NV accesses per
// vector, and the group's sum of squares is a shuffle reduction within it.
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
  __device__ static void load(const void* p, float (&x)[8]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  __device__ static void store(void* p, const float (&x)[8]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
};

__device__ __forceinline__ float group_sum(float v, int G) {
  for (int off = G >> 1; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float sigmoid_acc(float x) { return 1.0f / (1.0f + expf(-x)); }

// log(1 + e^x) without overflow: max(x, 0) + log1p(e^-|x|)
__device__ __forceinline__ float softplus_acc(float x) { return fmaxf(x, 0.0f) + log1pf(expf(-fabsf(x))); }

template <typename T, int NV>
__global__ __launch_bounds__(256) void k_prologue(const PrologueArgs a) {
  constexpr int EPV = Io<T>::EPV;
  const int G = a.group;
  const int lane_g = threadIdx.x & (G - 1);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H;
  const int64_t gstride = (int64_t)gridDim.x * (256 / G);
  const int nvec = a.hd / EPV;   // 16-byte accesses per vector
  for (int64_t g = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G; g < ngroups; g += gstride) {
    const int hh = (int)(g % a.H);
    const int64_t t = g / a.H;          // token b * L + l
    const int64_t b = t / a.L, l = t - b * a.L;
    const int64_t inst = b * a.H + hh;
    const bool kv = l < a.n_kv;
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      if (p > 0 && !kv) break;          // k, v exist for key tokens only
      const T* src = reinterpret_cast<const T*>(a.qkv) + ((t * 3 + p) * a.H + hh) * a.hd;
      float x[NV][8];
      float ss = 0.0f;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int vi = lane_g + j * G;
        if (vi < nvec) {
          Io<T>::load(src + vi * EPV, x[j]);
#pragma unroll
          for (int e = 0; e < EPV; ++e) {
            x[j][e] = x[j][e] * sigmoid_acc(x[j][e]);   // SiLU
            ss += x[j][e] * x[j][e];
          }
        }
      }
      float scale = 1.0f;
      if (p < 2) {                      // q / ||q||, k / ||k||; a zero vector stays zero
        ss = group_sum(ss, G);
        scale = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
      }
      T* dst = reinterpret_cast<T*>(p == 0 ? a.q : (p == 1 ? a.k : a.v)) +
               (inst * (p == 0 ? a.L : a.n_kv) + l) * a.hd;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int vi = lane_g + j * G;
        if (vi < nvec) {
#pragma unroll
          for (int e = 0; e < EPV; ++e) x[j][e] *= scale;
          Io<T>::store(dst + vi * EPV, x[j]);
        }
      }
    }
    if (kv)                             // learning rates: softplus(raw + bias)
      for (int r = lane_g; r < a.R; r += G)
        a.eta[(inst * a.n_kv + l) * a.R + r] = softplus_acc(a.lr_raw[(t * a.H + hh) * a.R + r] + a.lr_bias);
    if (kv && a.beta && lane_g == 0) a.beta[inst * a.n_kv + l] = sigmoid_acc(a.beta_raw[t * a.H + hh]);
  }
}

template <typename T, int NV>
__global__ __launch_bounds__(256) void k_rmsnorm_out(const RmsArgs a) {
  constexpr int EPV = Io<T>::EPV;
  const int G = a.group;
  const int lane_g = threadIdx.x & (G - 1);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H;
  const int64_t gstride = (int64_t)gridDim.x * (256 / G);
  const int nvec = a.hd / EPV;
  for (int64_t g = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G; g < ngroups; g += gstride) {
    // output order (b, l, h): consecutive groups write consecutive vectors
    const int hh = (int)(g % a.H);
    const int64_t t = g / a.H;
    const int64_t b = t / a.L, l = t - b * a.L;
    const T* src = reinterpret_cast<const T*>(a.o) + ((b * a.H + hh) * a.L + l) * a.hd;
    float x[NV][8];
    float ss = 0.0f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int vi = lane_g + j * G;
      if (vi < nvec) {
        Io<T>::load(src + vi * EPV, x[j]);
#pragma unroll
        for (int e = 0; e < EPV; ++e) ss += x[j][e] * x[j][e];
      }
    }
    ss = group_sum(ss, G);
    const float inv = 1.0f / sqrtf(ss / (float)a.hd + a.eps);
    T* dst = reinterpret_cast<T*>(a.y) + (t * a.H + hh) * a.hd;
    const float* w = a.weight ? a.weight + (int64_t)hh * a.hd : nullptr;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int vi = lane_g + j * G;
      if (vi < nvec) {
#pragma unroll
        for (int e = 0; e < EPV; ++e) x[j][e] *= inv * (w ? w[vi * EPV + e] : 1.0f);
        Io<T>::store(dst + vi * EPV, x[j]);
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

int64_t io_blocks(int64_t ngroups, int group) {
  const int64_t need = (ngroups * group + 255) / 256;
  return need < ((int64_t)1 << 20) ? need : ((int64_t)1 << 20);
}

template <template <typename, int> class KER, typename T, typename A>
hipError_t launch_nv(const A& a, int nv, int64_t blocks, hipStream_t s) {
  switch (nv) {
    case 1: KER<T, 1>::launch(a, blocks, s); break;
    case 2: KER<T, 2>::launch(a, blocks, s); break;
    case 4: KER<T, 4>::launch(a, blocks, s); break;
    case 8: KER<T, 8>::launch(a, blocks, s); break;
    default: KER<T, 16>::launch(a, blocks, s); break;
  }
  return hipGetLastError();
}

template <typename T, int NV> struct PrologueK {
  static void launch(const PrologueArgs& a, int64_t blocks, hipStream_t s) {
    k_prologue<T, NV><<<(unsigned)blocks, 256, 0, s>>>(a);
  }
};
template <typename T, int NV> struct RmsK {
  static void launch(const RmsArgs& a, int64_t blocks, hipStream_t s) {
    k_rmsnorm_out<T, NV><<<(unsigned)blocks, 256, 0, s>>>(a);
  }
};

// hd <= 4096: at most 1024 accesses of 16 bytes per vector, 16 per lane
int round_nv(int nv) { return nv <= 1 ? 1 : nv <= 2 ? 2 : nv <= 4 ? 4 : nv <= 8 ? 8 : 16; }

}  // namespace

hipError_t launch_prologue(PrologueArgs a, bool io_bf16, hipStream_t s) {
  int nv;
  io_shape(a.hd, io_bf16 ? 2 : 4, a.group, nv);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H;
  if (ngroups <= 0) return hipSuccess;
  const int64_t blocks = io_blocks(ngroups, a.group);
  nv = round_nv(nv);
  return io_bf16 ? launch_nv<PrologueK, __bf16>(a, nv, blocks, s) : launch_nv<PrologueK, float>(a, nv, blocks, s);
}

hipError_t launch_rmsnorm_out(RmsArgs a, bool io_bf16, hipStream_t s) {
  int nv;
  io_shape(a.hd, io_bf16 ? 2 : 4, a.group, nv);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H;
  if (ngroups <= 0) return hipSuccess;
  const int64_t blocks = io_blocks(ngroups, a.group);
  nv = round_nv(nv);
  return io_bf16 ? launch_nv<RmsK, __bf16>(a, nv, blocks, s) : launch_nv<RmsK, float>(a, nv, blocks, s);
}

}  // namespace lact
