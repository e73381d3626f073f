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

// Reverse of k_prologue, one group per (token, head) as there. With u =
// SiLU(x), s = sigmoid(x), SiLU'(x) = s + x s (1 - s); for q and k (y = u /
// |u|): du = dy / |u| - u (u . dy) / |u|^3 (zero for a zero u); for v: du = dy;
// dx = du SiLU'(x). Tokens past n_kv get zeros for k, v, the rates and beta.
template <typename T, int NV, typename IX>
__global__ __launch_bounds__(256) void k_prologue_bwd(const PrologueBwdArgs a) {
  constexpr int EPV = Io<T>::EPV;
  const int G = a.group;
  const int lane_g = threadIdx.x & (G - 1);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H;
  const int64_t gstride = (int64_t)gridDim.x * (256 / G);
  const int nvec = a.hd / EPV;
  for (int64_t g = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G; g < ngroups; g += gstride) {
    int hh;
    int64_t t, b, l;
    split_g<IX>(g, a.H, a.L, hh, t, b, l);
    const int64_t in = b * a.H + hh;
    const bool kv = l < a.n_kv;
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      const bool live = p == 0 || kv;
      const T* src = reinterpret_cast<const T*>(a.qkv) + ((t * 3 + p) * a.H + hh) * a.hd;
      const T* dsrc = live ? reinterpret_cast<const T*>(p == 0 ? a.dq : (p == 1 ? a.dk : a.dv)) +
                                 (in * (p == 0 ? a.L : a.n_kv) + l) * a.hd
                           : nullptr;
      float x[NV][8], dy[NV][8], up[NV][8];
      float ss = 0.0f, dot = 0.0f;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        if (!(live && lane_g + j * G < nvec)) continue;
        Io<T>::load(src + (lane_g + j * G) * EPV, x[j]);
        Io<T>::load(dsrc + (lane_g + j * G) * EPV, dy[j]);
#pragma unroll
        for (int e = 0; e < EPV; ++e) {
          const float z = x[j][e];
          const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z * -1.4426950408889634f));
          const float u = z * sg;
          up[j][e] = sg + u * (1.0f - sg);
          x[j][e] = u;
          ss += u * u;
          dot += u * dy[j][e];
        }
      }
      float inv = 1.0f, c = 0.0f;
      if (p < 2) {                    // the group shares `live`
        ss = group_sum(ss, G);
        dot = group_sum(dot, G);
        inv = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
        c = dot * inv * inv * inv;
      }
      T* dst = reinterpret_cast<T*>(a.dqkv) + ((t * 3 + p) * a.H + hh) * a.hd;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        if (lane_g + j * G >= nvec) continue;
        float o[8];
#pragma unroll
        for (int e = 0; e < EPV; ++e) o[e] = live ? (inv * dy[j][e] - c * x[j][e]) * up[j][e] : 0.0f;
        Io<T>::store(dst + (lane_g + j * G) * EPV, o);
      }
    }
    for (int r = lane_g; r < a.R; r += G) {   // d softplus(z) = sigmoid(z)
      const int64_t at = (t * a.H + hh) * a.R + r;
      a.dlr_raw[at] = kv ? a.deta[(in * a.n_kv + l) * a.R + r] * sigmoid_acc(a.lr_raw[at] + a.lr_bias) : 0.0f;
    }
    if (a.dbeta_raw && lane_g == 0) {
      const float bt = sigmoid_acc(a.beta_raw[t * a.H + hh]);
      a.dbeta_raw[t * a.H + hh] = kv ? a.dbeta[in * a.n_kv + l] * bt * (1.0f - bt) : 0.0f;
    }
  }
}

// Reverse of k_rmsnorm_out, one group per output vector (b, l, h): with r =
// 1 / sqrt(mean(o^2) + eps) and g = w dy, do = r g - (r^3 / hd) o (g . o);
// with dweight the vector's r goes to a.r for the weight's pass.
template <typename T, int NV, typename IX>
__global__ __launch_bounds__(256) void k_rmsnorm_out_bwd(const RmsBwdArgs a) {
  constexpr int EPV = Io<T>::EPV;
  const int G = a.group;
  const int lane_g = threadIdx.x & (G - 1);
  const int64_t ngroups = (int64_t)a.B * a.L * a.H;
  const int64_t gstride = (int64_t)gridDim.x * (256 / G);
  const int nvec = a.hd / EPV;
  for (int64_t g = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G; g < ngroups; g += gstride) {
    int hh;
    int64_t t, b, l;
    split_g<IX>(g, a.H, a.L, hh, t, b, l);
    const int64_t oo = ((b * a.H + hh) * a.L + l) * a.hd;
    float x[NV][8], gv[NV][8];
    float ss = 0.0f, dot = 0.0f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      if (lane_g + j * G >= nvec) continue;
      Io<T>::load(reinterpret_cast<const T*>(a.o) + oo + (lane_g + j * G) * EPV, x[j]);
      Io<T>::load(reinterpret_cast<const T*>(a.dy) + g * a.hd + (lane_g + j * G) * EPV, gv[j]);
      if (a.weight) {
        float w[8];
        Io<float>::load8(a.weight + (int64_t)hh * a.hd + (lane_g + j * G) * EPV, w, EPV);
#pragma unroll
        for (int e = 0; e < EPV; ++e) gv[j][e] *= w[e];
      }
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        ss += x[j][e] * x[j][e];
        dot += gv[j][e] * x[j][e];
      }
    }
    ss = group_sum(ss, G);
    dot = group_sum(dot, G);
    const float r = 1.0f / sqrtf(ss / (float)a.hd + a.eps);
    const float c = r * r * r * dot / (float)a.hd;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      if (lane_g + j * G >= nvec) continue;
      float o[8];
#pragma unroll
      for (int e = 0; e < EPV; ++e) o[e] = r * gv[j][e] - c * x[j][e];
      Io<T>::store(reinterpret_cast<T*>(a.d_o) + oo + (lane_g + j * G) * EPV, o);
    }
    if (a.dweight && lane_g == 0) a.r[g] = r;
  }
}

// The weight's cotangent, pass 1: workgroup (head h, 512 columns, split s)
// sums dy o r over its split's tokens into part[s][h][col]. Each lane owns 8
// columns (16-byte loads of bf16), each of the 4 waves every 4th token; the
// waves' sums are then added in order.
template <typename T>
__device__ __forceinline__ void load8c(const T* p, float (&x)[8]);
template <>
__device__ __forceinline__ void load8c<__bf16>(const __bf16* p, float (&x)[8]) { Io<__bf16>::load(p, x); }
template <>
__device__ __forceinline__ void load8c<float>(const float* p, float (&x)[8]) { Io<float>::load8(p, x, 8); }

template <typename T>
__global__ __launch_bounds__(256) void k_rms_dw_part(const RmsBwdArgs a, int nsplit, int64_t per) {
  __shared__ float red[4][512];
  const int cchunks = (a.hd + 511) / 512;
  const int sidx = blockIdx.x % nsplit;
  const int rest = blockIdx.x / nsplit;
  const int hh = rest / cchunks, c0 = (rest - hh * cchunks) * 512;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = c0 + 8 * lane;
  const bool on = col < a.hd;   // hd is a multiple of 8: a lane's columns are all in or all out
  const int64_t ntok = (int64_t)a.B * a.L;
  const int64_t t0 = sidx * per, t1 = t0 + per < ntok ? t0 + per : ntok;
  const T* dy = reinterpret_cast<const T*>(a.dy);
  const T* o = reinterpret_cast<const T*>(a.o);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (on) {
    for (int64_t t = t0 + w; t < t1; t += 4) {
      const int64_t b = t / a.L, l = t - b * a.L;
      float x[8], y[8];
      load8c<T>(dy + (t * a.H + hh) * a.hd + col, y);
      load8c<T>(o + ((b * a.H + hh) * a.L + l) * a.hd + col, x);
      const float rr = a.r[t * a.H + hh];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += y[e] * x[e] * rr;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[w][8 * lane + e] = acc[e];
  __syncthreads();
  if (w == 0 && on) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      a.part[((int64_t)sidx * a.H + hh) * a.hd + col + e] =
          (red[0][8 * lane + e] + red[1][8 * lane + e]) + (red[2][8 * lane + e] + red[3][8 * lane + e]);
  }
}

// Pass 2: dweight = the splits' partials summed in order.
__global__ __launch_bounds__(256) void k_rms_dw_sum(const float* part, float* dweight, int nsplit, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float acc = 0.0f;
  for (int sp = 0; sp < nsplit; ++sp) acc += part[(int64_t)sp * n + i];
  dweight[i] = acc;
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

template <typename T, int NV> struct PrologueBwdK {
  static void launch(const PrologueBwdArgs& a, hipStream_t s) {
    const int64_t n = (int64_t)a.B * a.L * a.H;
    const unsigned blocks = (unsigned)io_blocks(n, a.group);
    if (n < ((int64_t)1 << 31)) k_prologue_bwd<T, NV, uint32_t><<<blocks, 256, 0, s>>>(a);
    else k_prologue_bwd<T, NV, uint64_t><<<blocks, 256, 0, s>>>(a);
  }
};
template <typename T, int NV> struct RmsBwdK {
  static void launch(const RmsBwdArgs& a, hipStream_t s) {
    const int64_t n = (int64_t)a.B * a.L * a.H;
    const unsigned blocks = (unsigned)io_blocks(n, a.group);
    if (n < ((int64_t)1 << 31)) k_rmsnorm_out_bwd<T, NV, uint32_t><<<blocks, 256, 0, s>>>(a);
    else k_rmsnorm_out_bwd<T, NV, uint64_t><<<blocks, 256, 0, s>>>(a);
  }
};

// hd <= 4096: at most 1024 accesses of 16 bytes per vector, 16 per lane
int round_nv(int nv) { return nv <= 1 ? 1 : nv <= 2 ? 2 : nv <= 4 ? 4 : nv <= 8 ? 8 : 16; }

}  // namespace

hipError_t launch_prologue_bwd(PrologueBwdArgs a, bool io_bf16, hipStream_t s) {
  int nv;
  io_shape(a.hd, io_bf16 ? 2 : 4, a.group, nv);
  if ((int64_t)a.B * a.L * a.H <= 0) return hipSuccess;
  nv = round_nv(nv);
  return io_bf16 ? launch_nv<PrologueBwdK, __bf16>(a, nv, s) : launch_nv<PrologueBwdK, float>(a, nv, s);
}

// Token splits of the weight's pass: about 2048 workgroups in all.
int rms_dw_splits(int B, int64_t L, int H, int hd) {
  const int64_t ntok = (int64_t)B * L, tiles = (int64_t)H * ((hd + 511) / 512);
  int64_t sp = (2048 + tiles - 1) / tiles;
  if (sp > 256) sp = 256;
  if (sp > ntok) sp = ntok;
  return (int)(sp < 1 ? 1 : sp);
}

hipError_t launch_rmsnorm_out_bwd(RmsBwdArgs a, bool io_bf16, hipStream_t s) {
  int nv;
  io_shape(a.hd, io_bf16 ? 2 : 4, a.group, nv);
  if ((int64_t)a.B * a.L * a.H <= 0) return hipSuccess;
  nv = round_nv(nv);
  hipError_t e = io_bf16 ? launch_nv<RmsBwdK, __bf16>(a, nv, s) : launch_nv<RmsBwdK, float>(a, nv, s);
  if (e != hipSuccess || !a.dweight) return e;
  const int nsplit = rms_dw_splits(a.B, a.L, a.H, a.hd);
  const int64_t ntok = (int64_t)a.B * a.L, per = (ntok + nsplit - 1) / nsplit;
  const int64_t blocks = (int64_t)nsplit * a.H * ((a.hd + 511) / 512);
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  if (io_bf16) k_rms_dw_part<__bf16><<<(unsigned)blocks, 256, 0, s>>>(a, nsplit, per);
  else k_rms_dw_part<float><<<(unsigned)blocks, 256, 0, s>>>(a, nsplit, per);
  const int64_t n = (int64_t)a.H * a.hd;
  k_rms_dw_sum<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(a.part, a.dweight, nsplit, n);
  return hipGetLastError();
}

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
