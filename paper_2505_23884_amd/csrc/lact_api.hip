// Host side of the C ABI: validation, workspace layout, the chunk schedule
// and kernel timing. Everything in here runs on the host; all arithmetic of
// the path runs in lact_kernels.hip.
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "lact.h"
#include "lact_internal.h"

// Scratch memory of lact_forward_noalloc (its workspace, for callers that
// cannot allocate): one copy per device, loaded with the library's device
// code and held until the process ends. In host code `scratch` is only the
// symbol's stand-in; its device address comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[LACT_NOALLOC_SCRATCH_BYTES];

namespace lact {
namespace {

thread_local char g_hip_err[256] = "";

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Shape-derived plan shared by lact_workspace_bytes and lact_forward.
struct Plan {
  int BH, d, h;
  bool bf16;
  int esz;
  int es;             // floats of eta per token (1, or 3 with per-matrix rates)
  bool linear;        // linear fast weight: one d x d matrix per instance (h == d)
  int nmat;           // fast-weight matrices per instance (3 or 1)
  int64_t C;          // tokens of the largest chunk (0 when n_kv == 0)
  int64_t cap;        // rows of the applied-hidden buffer
  int nsplit;         // split-K ways of the gradient contraction
  int64_t split_len;  // tokens per split
  bool fused;         // gradient and weight update in one kind (BWD_GRAD_UPD)
  bool narrow;        // narrow tile shapes of both launches (16-bit, d <= 128)
  bool ns_out;        // a chunk's output tiles run with its fused Newton-Schulz
  bool muon;
  bool tile_sums;     // Muon without split: the gradient tiles leave the sums of squares
  int t13, t2;        // gradient tiles per matrix (W1 or W3; W2 or the linear W)
  bool ns_fp16;       // Newton-Schulz operand copies in fp16 (bf16 I/O) or fp32
  int ns_esz;
  int m;              // Newton-Schulz Gram size min(d, h)
  int ns_bps;         // blocks of kNsBlockElems per gradient
  // workspace offsets (bytes)
  size_t off_wb[3], off_wb2[3], off_hq, off_upd[3], off_step, off_bbar, total;
  size_t off_y32, off_yb[2], off_ab, off_a2, off_bb, off_ss;
};

int check_desc(const lact_desc* d) {
  if (!d) return LACT_EINVAL;
  if (d->B < 1 || d->H < 1) return LACT_EINVAL;
  if (d->n_kv < 0 || d->n_q < d->n_kv || d->chunk < 1) return LACT_EINVAL;
  if (d->order != LACT_APPLY_THEN_UPDATE && d->order != LACT_UPDATE_THEN_APPLY) return LACT_EINVAL;
  if (d->use_muon != 0 && d->use_muon != 1) return LACT_EINVAL;
  if (d->ns_steps < 0 || d->ns_steps > 16) return LACT_EINVAL;
  if (d->io_dtype != LACT_IO_BF16 && d->io_dtype != LACT_IO_FP32) return LACT_EINVAL;
  if (d->eta_per_matrix != 0 && d->eta_per_matrix != 1) return LACT_EINVAL;
  if (d->fast_weight != LACT_FW_SWIGLU && d->fast_weight != LACT_FW_LINEAR) return LACT_EINVAL;
  // the linear fast weight is one d x d matrix with one learning rate per token
  if (d->fast_weight == LACT_FW_LINEAR && (d->h != d->d || d->eta_per_matrix)) return LACT_EINVAL;
  if (d->d < 1 || d->h < 1) return LACT_EINVAL;
  if (d->d % 8 || d->h % 8 || d->d > kMaxDim || d->h > kMaxDim) return LACT_EUNSUPPORTED;
  // 16-bit MFMA tiles take K in whole steps of 32 along d and h
  if (d->io_dtype == LACT_IO_BF16 && (d->d % 32 || d->h % 32)) return LACT_EUNSUPPORTED;
  if ((int64_t)d->B * d->H > (1 << 20)) return LACT_EUNSUPPORTED;
  if (d->n_q > ((int64_t)1 << 40)) return LACT_EUNSUPPORTED;
  // Every launch's grid must fit the 32-bit block count: bounds with the
  // smallest tile edge (128) for the contractions, the most splits for the
  // gradient, one wave per weight row for the update and 4096-element blocks
  // for the Newton-Schulz prologue (such sizes exceed any GPU's memory long
  // before they reach these bounds, but the check keeps the launches exact).
  const int64_t BH = (int64_t)d->B * d->H, mx = std::max(d->d, d->h);
  const int64_t C = std::min<int64_t>(d->chunk, d->n_kv);
  const int64_t L = std::max<int64_t>(std::max<int64_t>(C, 1), std::min<int64_t>(d->n_q, C + std::max<int64_t>(C, 65536)));
  const int64_t t = (mx + 127) / 128;
  const double most = std::max({(double)BH * t * ((L + 127) / 128) * 2.0, (double)BH * t * t * 2.0 * kMaxSplit,
                                (double)BH * 3.0 * mx, (double)BH * 3.0 * ((mx * mx + 4095) / 4096)});
  if (most > 2147483647.0) return LACT_EUNSUPPORTED;
  return LACT_OK;
}

Plan make_plan(const lact_desc* dsc, bool allow_fused = true) {
  Plan p{};
  p.BH = dsc->B * dsc->H;
  p.d = dsc->d;
  p.h = dsc->h;
  p.bf16 = dsc->io_dtype == LACT_IO_BF16;
  p.esz = p.bf16 ? 2 : 4;
  p.es = dsc->eta_per_matrix ? 3 : 1;
  p.linear = dsc->fast_weight == LACT_FW_LINEAR;
  p.nmat = p.linear ? 1 : 3;
  p.C = std::min<int64_t>(dsc->chunk, dsc->n_kv);
  p.narrow = p.bf16 && p.d <= 128;
  // Small matrices with Muon (one fused Newton-Schulz workgroup each) and the
  // narrow tile shapes: the output tiles of a chunk's apply run in the
  // Newton-Schulz launch, on the CUs its one workgroup per matrix leaves idle,
  // instead of beside the gradient tiles; the update writes the other set of
  // operand copies. (Video: 4.39 -> 4.29 ms per step. The gradient tiles then
  // have the second launch to themselves; three or four splits instead of two
  // did not pay: the Newton-Schulz workgroups sum the partials.)
  p.ns_out = p.narrow && dsc->use_muon && !p.linear && std::min(p.d, p.h) <= kNsFusedM &&
             std::max(p.d, p.h) <= kNsFusedN;
  const int64_t tail = dsc->n_q - dsc->n_kv;
  // The applied-hidden buffer holds one chunk plus (bounded) tail rows so that
  // update-then-apply can apply its last chunk together with the tail.
  p.cap = std::min<int64_t>(dsc->n_q, p.C + std::min<int64_t>(tail, std::max<int64_t>(p.C, 65536)));
  if (p.cap < 1) p.cap = 1;
  // Split-K of the gradient contraction (fp32 partials, summed by the weight
  // update). Each split adds a full write and read of 3*d*h fp32 per instance,
  // worth about 500 tokens of the gradient's own work, so short chunks (the
  // LM workload's 2048) split only when the gradient tiles alone would leave
  // most of the chip idle (measured: 2 splits cost 8% there; on the video
  // shape 4 splits instead of 2 cost 7%). Long chunks
  // (NVS: one chunk of up to 1M tokens) take the split count, with splits of
  // at least 1024 tokens, that minimises the makespan of equal blocks over the
  // 256 CUs, rounds(tiles * ns) / ns, plus a small cost per split (its
  // partial's write and read against a block of the whole chunk: NVS 1M takes
  // 14 splits, 3 full rounds, 1% faster than 9 splits in 2 uneven rounds).
  // Lengths are a multiple of 32.
  const TileShape g13 = bwd_tile(BWD_GRAD13, p.bf16, p.narrow), g2 = bwd_tile(BWD_GRAD2, p.bf16, p.narrow);
  const int64_t tiles = (int64_t)p.BH * ((p.linear ? 0 : cdiv(p.h, g13.rows) * cdiv(p.d, g13.cols)) +
                                         cdiv(p.d, g2.rows) * cdiv(p.h, g2.cols));
  // The gradient and update kind (below) needs an unsplit gradient; it pays
  // when its row tiles cover at least half the chip and, for long chunks, when
  // apply tiles share the launch (apply-then-update, or more than one chunk)
  // and take the CUs the row tiles leave.
  const int upd_cols = grad_upd_tile().cols;
  const bool upd_shape = allow_fused && p.bf16 && !p.linear && !dsc->use_muon && p.d > 256 && p.h > 256 &&
                         p.d <= upd_cols && p.h <= upd_cols;
  const bool apply_alongside = dsc->order == LACT_APPLY_THEN_UPDATE || dsc->n_kv > p.C;
  int64_t ns;
  if (upd_shape && tiles >= 128 && (p.C < 8192 || apply_alongside)) {
    ns = 1;
  } else if (p.C >= 8192) {
    const int64_t top = std::min<int64_t>(kMaxSplit, std::max<int64_t>(1, p.C / 1024));
    ns = 1;
    double best = 1e30;
    for (int64_t t = 1; t <= top; ++t) {
      const double cost = (double)cdiv(tiles * t, 256) / (double)t + 0.0002 * (double)t;
      if (cost < best - 1e-12) {
        best = cost;
        ns = t;
      }
    }
  } else {
    ns = std::max<int64_t>(1, cdiv(128, tiles));
    ns = std::min<int64_t>(ns, std::max<int64_t>(1, p.C / 256));
  }
  ns = std::min<int64_t>(ns, kMaxSplit);
  p.split_len = std::max<int64_t>(32, cdiv(cdiv(std::max<int64_t>(p.C, 1), ns), 32) * 32);
  p.nsplit = (int)std::max<int64_t>(1, cdiv(std::max<int64_t>(p.C, 1), p.split_len));
  // The gradient and the weight update (with momentum or without) run as one
  // kind (BWD_GRAD_UPD) when a tile holds whole rows of W1, W2 and W3
  // (256 < d, h <= 512: narrower rows would leave most of the tile empty), the
  // gradient is not split and no Newton-Schulz step sits between the two. The
  // bf16 operand copies then alternate between two buffers: the apply tiles
  // of the same launch still read the pre-update W2.
  p.fused = upd_shape && p.nsplit == 1;
  const size_t dh = (size_t)p.d * p.h;
  size_t o = 0;
  for (int m = 0; m < 3; ++m) {
    p.off_wb[m] = o;
    if (p.bf16 && m < p.nmat) o = align_up(o + (size_t)p.BH * dh * 2);
  }
  for (int m = 0; m < 3; ++m) {
    p.off_wb2[m] = o;
    if (p.fused || p.ns_out) o = align_up(o + (size_t)p.BH * dh * 2);
  }
  // linear: no applied hidden (the apply is one product); one update buffer (eta k)
  p.off_hq = o;
  if (!p.linear) o = align_up(o + (size_t)p.BH * p.cap * p.h * p.esz);
  for (int m = 0; m < 3; ++m) {
    p.off_upd[m] = o;
    if (m < p.nmat) o = align_up(o + (size_t)p.BH * std::max<int64_t>(p.C, 1) * p.h * p.esz);
  }
  p.off_step = o;
  o = align_up(o + (size_t)p.nsplit * p.BH * p.nmat * dh * 4);
  // chunk-mean momentum factors of up to kBetaBatch chunks (momentum entry
  // point only; reserved always so both entry points share one size)
  p.off_bbar = o;
  o = align_up(o + (size_t)p.BH * kBetaBatch * 4);
  p.muon = dsc->use_muon != 0;
  p.m = std::min(p.d, p.h);
  p.ns_bps = (int)cdiv((int64_t)dh, kNsBlockElems);
  p.t13 = p.linear ? 0 : (int)(cdiv(p.h, g13.rows) * cdiv(p.d, g13.cols));
  p.t2 = (int)(cdiv(p.d, g2.rows) * cdiv(p.h, g2.cols));
  // Without split the sums of squares that Newton-Schulz normalises by come
  // from the gradient tiles' epilogues (one entry per tile), and the scaling
  // reads the gradient directly: no separate pass over it (momentum keeps the
  // pass, which also advances the state). Small matrices (one fused
  // Newton-Schulz workgroup each) take their norm in that workgroup instead.
  p.ns_fp16 = p.bf16;
  const bool ns_small = p.ns_fp16 && p.m <= kNsFusedM && std::max(p.d, p.h) <= kNsFusedN;
  p.tile_sums = p.muon && p.nsplit == 1 && p.t13 <= p.ns_bps && p.t2 <= p.ns_bps && !ns_small;
  p.ns_esz = p.ns_fp16 ? 2 : 4;
  if (p.muon) {
    const size_t slots = (size_t)p.BH * p.nmat, mm = (size_t)p.m * p.m;
    p.off_y32 = o;
    o = align_up(o + slots * dh * 4);
    for (int i = 0; i < 2; ++i) {
      p.off_yb[i] = o;
      o = align_up(o + slots * dh * p.ns_esz);
    }
    p.off_ab = o;
    o = align_up(o + slots * mm * p.ns_esz);
    p.off_a2 = o;
    o = align_up(o + slots * mm * p.ns_esz);
    p.off_bb = o;
    o = align_up(o + slots * mm * p.ns_esz);
    p.off_ss = o;
    o = align_up(o + slots * p.ns_bps * 4);
  }
  p.total = o;
  return p;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15) != 0; }

// ---------------------------------------------------------------- timing
struct TimedLaunch {
  hipEvent_t a, b;
  int kclass;
  double flops;
};
struct Timing {
  bool enabled = false;
  std::vector<hipEvent_t> pool;
  std::vector<TimedLaunch> pending;
  int64_t launches[LACT_KCLASS_COUNT] = {};
  double ms[LACT_KCLASS_COUNT] = {};
  double flops[LACT_KCLASS_COUNT] = {};
};
Timing g_timing;
constexpr size_t kMaxTimed = 65536;

hipEvent_t pool_event() {
  if (!g_timing.pool.empty()) {
    hipEvent_t e = g_timing.pool.back();
    g_timing.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

int record_hip(hipError_t e) {
  if (e == hipSuccess) return LACT_OK;
  snprintf(g_hip_err, sizeof g_hip_err, "%s", hipGetErrorString(e));
  return LACT_EHIP;
}

// Runs `launch` on `s`, bracketed by events when timing is enabled.
template <class F>
int timed(int kclass, double flops, hipStream_t s, F&& launch) {
  hipEvent_t ea = nullptr, eb = nullptr;
  const bool t = g_timing.enabled && g_timing.pending.size() < kMaxTimed;
  if (t) {
    ea = pool_event();
    eb = pool_event();
    if (ea && eb && hipEventRecord(ea, s) != hipSuccess) ea = nullptr;
  }
  int rc = record_hip(launch());
  if (t && ea && eb && hipEventRecord(eb, s) == hipSuccess)
    g_timing.pending.push_back({ea, eb, kclass, flops});
  if (rc == LACT_OK && getenv("LACT_SYNC") && getenv("LACT_SYNC")[0] == '1')
    rc = record_hip(hipStreamSynchronize(s));
  return rc;
}

// ---------------------------------------------------------------- schedule
struct Ctx {
  const lact_desc* dsc;
  Plan p;
  const uint8_t *q, *k, *v;
  const float* eta;
  float* W[3];
  uint8_t* o;
  uint8_t* ws;
  hipStream_t s;
  Operand wop[3];   // operand copies of W1, W2, W3 (bf16 copies or the fp32 state)
  void* wb[2][3];   // the two sets of bf16 copies (the second with BWD_GRAD_UPD)
  int wset;         // the set wop points at
  bool ns_updated;  // the last Newton-Schulz step has also applied the weight update
  const float* beta;   // momentum: per-token factor [BH][n_kv], or nullptr
  float* M[3];         // momentum state (with beta)
  int64_t chunk_idx;   // index of the chunk being updated
  BwdArgs out_pending{};   // with ns_out: the output tiles the next Newton-Schulz launch runs
  double out_flops = 0.0;
  bool has_out = false;
  bool grad_only = false;   // update_chunk stops after the gradient partials (the backward's own update follows)
  void* keep[3] = {};       // or nullptr: where the key forward also writes Z1, Z3 and D (FwdSeg::keep)
  int64_t keep_inst = 0;
  const float* Wsrc[3] = {};   // where the update reads the state (nullptr: W, in place)
};

// Momentum factor of the current chunk for instance 0 (stride kBetaBatch).
const float* bbar_of(const Ctx& c) {
  return reinterpret_cast<const float*>(c.ws + c.p.off_bbar) + c.chunk_idx % kBetaBatch;
}

Operand op(const void* base, int64_t ld, int64_t inst) { return Operand{base, ld, inst}; }

// Applies the current fast weights to query rows [s0, s1), in pieces that fit.
int apply_rows(Ctx& c, int64_t s0, int64_t s1) {
  const Plan& p = c.p;
  if (p.linear) {   // o = W q: one contraction over d per piece of rows
    for (int64_t a = s0; a < s1; a += 65536) {   // bounds the tile count of a launch
      const int64_t n = std::min<int64_t>(65536, s1 - a);
      BwdArgs b{};
      BwdSeg& o = b.seg[0];
      o.kind = BWD_OUT;
      o.tiles_m = (int)cdiv(p.d, bwd_tile(BWD_OUT, p.bf16, p.narrow).rows);
      o.tiles_n = (int)cdiv(n, bwd_tile(BWD_OUT, p.bf16, p.narrow).cols);
      o.nsplit = 1;
      o.nblocks = p.BH * o.tiles_m * o.tiles_n;
      o.rows = n;
      o.a0 = op(c.q + a * p.d * p.esz, p.d, c.dsc->n_q * p.d);
      o.b0 = c.wop[0];
      o.out = c.o + a * p.d * p.esz;
      o.out_inst = c.dsc->n_q * p.d;
      b.nseg = 1;
      b.total_blocks = o.nblocks;
      b.d = p.d;
      b.h = p.d;
      b.narrow = p.narrow;
      const int rc = timed(LACT_KCLASS_BWD, 2.0 * p.BH * n * p.d * p.d, c.s,
                           [&] { return launch_bwd(b, p.bf16, c.s); });
      if (rc) return rc;
    }
    return LACT_OK;
  }
  for (int64_t a = s0; a < s1; a += p.cap) {
    const int64_t n = std::min<int64_t>(p.cap, s1 - a);
    FwdArgs f{};
    FwdSeg& g = f.seg[0];
    g.kind = FWD_APPLY;
    g.tiles_m = (int)cdiv(p.h, fwd_tile(FWD_APPLY, p.bf16, p.narrow).rows);
    g.tiles_n = (int)cdiv(n, fwd_tile(FWD_APPLY, p.bf16, p.narrow).cols);
    g.nblocks = p.BH * g.tiles_m * g.tiles_n;
    g.rows = n;
    g.a0 = op(c.q + a * p.d * p.esz, p.d, c.dsc->n_q * p.d);
    g.out0 = c.ws + p.off_hq;
    g.out_inst = p.cap * p.h;
    f.nseg = 1;
    f.total_blocks = g.nblocks;
    f.d = p.d;
    f.h = p.h;
    f.narrow = p.narrow;
    f.w1 = c.wop[0];
    f.w2 = c.wop[1];
    f.w3 = c.wop[2];
    const double fl1 = 4.0 * p.BH * n * p.d * p.h;
    int rc = timed(LACT_KCLASS_FWD, fl1, c.s, [&] { return launch_fwd(f, p.bf16, c.s); });
    if (rc) return rc;
    BwdArgs b{};
    BwdSeg& o = b.seg[0];
    o.kind = BWD_OUT;
    o.tiles_m = (int)cdiv(p.d, bwd_tile(BWD_OUT, p.bf16, p.narrow).rows);
    o.tiles_n = (int)cdiv(n, bwd_tile(BWD_OUT, p.bf16, p.narrow).cols);
    o.nsplit = 1;
    o.nblocks = p.BH * o.tiles_m * o.tiles_n;
    o.rows = n;
    o.a0 = op(c.ws + p.off_hq, p.h, p.cap * p.h);
    o.b0 = c.wop[1];
    o.out = c.o + a * p.d * p.esz;
    o.out_inst = c.dsc->n_q * p.d;
    b.nseg = 1;
    b.total_blocks = o.nblocks;
    b.d = p.d;
    b.h = p.h;
    b.narrow = p.narrow;
    rc = timed(LACT_KCLASS_BWD, 2.0 * p.BH * n * p.d * p.h, c.s, [&] { return launch_bwd(b, p.bf16, c.s); });
    if (rc) return rc;
  }
  return LACT_OK;
}

void use_wset(Ctx& c, int set);

// Muon (§3.2; App. A): Newton-Schulz on the three summed gradients of every
// instance, in their stored orientation; leaves NS(P) in the fp32 iterate.
int newton_schulz(Ctx& c) {
  const Plan& p = c.p;
  const int64_t dh = (int64_t)p.d * p.h;
  NsPrepArgs pa{};
  pa.part = reinterpret_cast<const float*>(c.ws + p.off_step);
  pa.nsplit = p.nsplit;
  pa.part_split = (int64_t)p.BH * p.nmat * dh;
  pa.Y32 = reinterpret_cast<float*>(c.ws + p.off_y32);
  pa.spi = p.nmat;
  pa.sumsq = reinterpret_cast<float*>(c.ws + p.off_ss);
  pa.nslots = p.BH * p.nmat;
  pa.dh = dh;
  pa.blocks_per_slot = p.ns_bps;
  if (c.beta) {
    for (int j = 0; j < p.nmat; ++j) pa.M[j] = c.M[j];
    pa.bbar = bbar_of(c);
    pa.bbar_stride = kBetaBatch;
  }
  int rc = LACT_OK;
  const int m = p.m, d = p.d, h = p.h;
  // small matrices: the fused kernel normalises the gradient itself (after
  // the momentum step of k_ns_prep, if any)
  const bool fused = p.ns_fp16 && m <= kNsFusedM && std::max(d, h) <= kNsFusedN;
  if (p.tile_sums && !c.beta && !fused) {
    pa.src = reinterpret_cast<const float*>(c.ws + p.off_step);
    pa.sum_n[0] = p.linear ? p.t2 : p.t13;
    pa.sum_n[1] = p.t2;
    pa.sum_n[2] = p.t13;
  } else if (!fused || c.beta) {
    rc = timed(LACT_KCLASS_NS, 0.0, c.s, [&] { return launch_ns_prep(pa, c.s); });
    if (rc) return rc;
  }
  if (!fused) {
    rc = timed(LACT_KCLASS_NS, 0.0, c.s,
               [&] { return launch_ns_scale(pa, c.ws + p.off_yb[0], p.ns_fp16, kNsEps, c.s); });
    if (rc) return rc;
  }
  // segment 0: W1 and W3 stored h x d; segment 1: W2 stored d x h
  // (linear: one segment, the d x d matrix)
  const int rows[2] = {h, d}, cols[2] = {d, h};
  const int nseg = p.linear ? 1 : 2;
  auto group_of = [&](int g) { return p.linear ? 1 : (g == 0 ? 2 : 1); };
  auto slot_of = [&](int g) { return p.linear ? 0 : (g == 0 ? 0 : 1); };
  if (fused) {
    // small matrices: every step of one matrix in one workgroup, both
    // groups (W1 and W3, W2) in one launch
    const int n = std::max(d, h);
    NsFusedArgs fs[2]{};
    double fl = 0.0;
    for (int g = 0; g < nseg; ++g) {
      NsFusedArgs& f = fs[g];
      f.spi = p.nmat;
      f.ystride = dh;
      f.group = group_of(g);
      f.slot_off[0] = slot_of(g);
      f.slot_off[1] = 2;
      f.rows = rows[g];
      f.cols = cols[g];
      f.nblocks = p.BH * f.group;
      f.steps = c.dsc->ns_steps;
      f.ca = kNsA;
      f.cb = kNsB;
      f.cc = kNsC;
      // the summed gradient: the split partials, or the momentum state's
      // iterate that k_ns_prep left in Y32
      f.src = c.beta ? pa.Y32 : pa.part;
      f.nsplit = c.beta ? 1 : p.nsplit;
      f.part_split = pa.part_split;
      f.eps = kNsEps;
      // and the weight update (no separate update launch follows); with
      // output tiles in the launch, the copies go to the other set
      for (int j = 0; j < p.nmat; ++j) {
        f.W[j] = c.W[j];
        f.Wb[j] = c.wb[c.has_out ? c.wset ^ 1 : c.wset][j];
      }
      fl += (double)f.steps * f.nblocks * (4.0 * m * m * n + 2.0 * m * m * m);
    }
    if (c.has_out) {
      if (nseg != 2) return LACT_EUNSUPPORTED;
      c.has_out = false;
      rc = timed(LACT_KCLASS_NS, fl + c.out_flops, c.s,
                 [&] { return launch_ns_fused_pair_out(fs[0], fs[1], c.out_pending, c.s); });
      if (rc) return rc;
      use_wset(c, c.wset ^ 1);   // the next launches read the new copies
    } else {
      rc = timed(LACT_KCLASS_NS, fl, c.s, [&] {
        return nseg == 2 ? launch_ns_fused_pair(fs[0], fs[1], c.s) : launch_ns_fused(fs[0], c.s);
      });
      if (rc) return rc;
    }
    c.ns_updated = true;
    return LACT_OK;
  }
  const int64_t mm = (int64_t)m * m;
  // Gram matrices larger than 128 (16-bit operands): the update product in
  // 256 x 256 tiles; the Gram and polynomial products, which are symmetric,
  // in 128 x 128 tiles of the upper triangle only (10 of 16 at m = 512), two
  // workgroups per CU. Smaller matrices: 128 x 128 tiles throughout.
  const bool big = p.ns_fp16 && m > 128;
  // Square matrices (d == h) of side up to 512 with 16-bit operands: the last
  // step's update product and the weight update run as one launch
  // (k_ns_final), which writes W and its copy instead of the iterate.
  const bool fuse_last = p.ns_fp16 && d == h && m <= ns_final_tile().cols && c.dsc->ns_steps >= 1;
  for (int t = 0; t < c.dsc->ns_steps; ++t) {
    NsArgs a{};
    a.Y32 = pa.Y32;
    a.spi = p.nmat;
    a.Yin = c.ws + p.off_yb[t & 1];
    // the last step's operand copy would never be read: only the fp32 iterate
    a.Yout = t + 1 < c.dsc->ns_steps ? (void*)(c.ws + p.off_yb[(t + 1) & 1]) : nullptr;
    a.Ab = c.ws + p.off_ab;
    a.A2b = c.ws + p.off_a2;
    a.Bb = c.ws + p.off_bb;
    a.ystride = dh;
    a.astride = mm;
    a.m = m;
    a.ca = kNsA;
    a.cb = kNsB;
    a.cc = kNsC;
    a.nseg = nseg;
    for (int phase = 0; phase < 3; ++phase) {
      if (phase == 2 && fuse_last && t + 1 == c.dsc->ns_steps) {
        NsFinalArgs f{};
        f.Bb = c.ws + p.off_bb;
        f.Yin = c.ws + p.off_yb[t & 1];
        f.Y32 = pa.Y32;
        for (int j = 0; j < p.nmat; ++j) {
          f.W[j] = c.W[j];
          f.Wb[j] = c.wb[c.wset][j];
        }
        f.spi = p.nmat;
        f.m = m;
        f.ystride = dh;
        f.astride = mm;
        f.nblocks = (int)(p.BH * p.nmat * cdiv(m, ns_final_tile().rows));
        f.ca = kNsA;
        const double fl = 2.0 * p.BH * p.nmat * (double)m * m * m;
        rc = timed(LACT_KCLASS_NS, fl, c.s, [&] { return launch_ns_final(f, c.s); });
        if (rc) return rc;
        c.ns_updated = true;
        continue;
      }
      a.total_blocks = 0;
      double fl = 0.0;
      const bool tri = big && phase < 2;
      const bool bigp = big && !tri;
      for (int g = 0; g < nseg; ++g) {
        NsSeg& sg = a.seg[g];
        sg.tri = tri;
        sg.group = group_of(g);
        sg.slot_off[0] = slot_of(g);
        sg.slot_off[1] = 2;
        sg.ldy = cols[g];
        const bool wide = rows[g] <= cols[g];
        const int n = std::max(rows[g], cols[g]);
        if (phase == 0) {
          sg.kind = wide ? NS_GRAM_K : NS_GRAM_MN;
          sg.M = sg.N = m;
          sg.K = n;
        } else if (phase == 1) {
          sg.kind = NS_POLY;
          sg.M = sg.N = sg.K = m;
        } else {
          // tile space of the update: rows = columns of Y, columns = rows of Y
          sg.kind = wide ? NS_UPD_BY : NS_UPD_YB;
          sg.M = cols[g];
          sg.N = rows[g];
          sg.K = m;
        }
        const TileShape ts = ns_tile(p.ns_fp16, bigp);
        sg.tiles_m = (int)cdiv(sg.M, ts.rows);
        sg.tiles_n = (int)cdiv(sg.N, ts.cols);
        sg.nblocks = p.BH * sg.group * (tri ? sg.tiles_m * (sg.tiles_m + 1) / 2 : sg.tiles_m * sg.tiles_n);
        a.total_blocks += sg.nblocks;
        // FLOPs of the tiles computed (the triangle's: its off-diagonal tiles
        // are written twice but computed once)
        double area = (double)sg.M * sg.N;
        if (tri) {
          area = 0.0;
          for (int ti = 0; ti < sg.tiles_m; ++ti)
            for (int tj = ti; tj < sg.tiles_m; ++tj)
              area += (double)std::min(ts.rows, sg.M - ti * ts.rows) * std::min(ts.cols, sg.N - tj * ts.cols);
        }
        fl += 2.0 * p.BH * sg.group * area * sg.K;
      }
      rc = timed(LACT_KCLASS_NS, fl, c.s, [&] { return launch_ns(a, p.ns_fp16, bigp, c.s); });
      if (rc) return rc;
    }
  }
  return LACT_OK;
}

int finish_update(Ctx& c);
int update_chunk_linear(Ctx& c, int64_t s0, int64_t s1, bool apply_too);

// Gradient segments of a Muon update without split or momentum write their
// tiles' sums of squares (GRAD2 for matrix j2: W2, or the linear W).
void set_tile_sums(const Ctx& c, BwdSeg& g, int j2) {
  if (!c.p.tile_sums || c.beta) return;
  g.sumsq = reinterpret_cast<float*>(c.ws + c.p.off_ss);
  g.sumsq_stride = c.p.ns_bps;
  g.sumsq_j = j2;
  g.spi = c.p.nmat;
}

// Points the operand views at bf16 copy set `set`.
void use_wset(Ctx& c, int set) {
  const int64_t dh = (int64_t)c.p.d * c.p.h;
  c.wset = set;
  c.wop[0] = op(c.wb[set][0], c.p.d, dh);
  c.wop[1] = op(c.wb[set][1], c.p.h, dh);
  c.wop[2] = op(c.wb[set][2], c.p.d, dh);
}

// One update on key rows [s0, s1); with apply_too, the same launches also
// apply the current (pre-update) weights to query rows [s0, s1).
int update_chunk(Ctx& c, int64_t s0, int64_t s1, bool apply_too) {
  if (c.p.linear) return update_chunk_linear(c, s0, s1, apply_too);
  const Plan& p = c.p;
  const int64_t n = s1 - s0;
  const int64_t dh = (int64_t)p.d * p.h;
  FwdArgs f{};
  int ns = 0;
  {
    FwdSeg& g = f.seg[ns++];
    g.kind = FWD_UPDATE;
    g.tiles_m = (int)cdiv(p.h, fwd_tile(FWD_UPDATE, p.bf16, p.narrow).rows);
    g.tiles_n = (int)cdiv(n, fwd_tile(FWD_UPDATE, p.bf16, p.narrow).cols);
    g.nblocks = p.BH * g.tiles_m * g.tiles_n;
    g.rows = n;
    g.a0 = op(c.k + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);
    g.a1 = op(c.v + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);
    g.out1 = c.ws + p.off_upd[0];
    g.out2 = c.ws + p.off_upd[1];
    g.out3 = c.ws + p.off_upd[2];
    g.out_inst = p.C * p.h;
    g.eta = c.eta + s0 * p.es;
    g.eta_inst = c.dsc->n_kv * p.es;
    g.eta_stride = p.es;
    for (int m = 0; m < 3; ++m) g.keep[m] = c.keep[m];
    g.keep_inst = c.keep_inst;
  }
  if (apply_too) {
    FwdSeg& g = f.seg[ns++];
    g.kind = FWD_APPLY;
    g.tiles_m = (int)cdiv(p.h, fwd_tile(FWD_APPLY, p.bf16, p.narrow).rows);
    g.tiles_n = (int)cdiv(n, fwd_tile(FWD_APPLY, p.bf16, p.narrow).cols);
    g.nblocks = p.BH * g.tiles_m * g.tiles_n;
    g.rows = n;
    g.a0 = op(c.q + s0 * p.d * p.esz, p.d, c.dsc->n_q * p.d);
    g.out0 = c.ws + p.off_hq;
    g.out_inst = p.cap * p.h;
  }
  f.nseg = ns;
  f.total_blocks = f.seg[0].nblocks + (ns > 1 ? f.seg[1].nblocks : 0);   // long tiles first
  f.d = p.d;
  f.h = p.h;
  f.narrow = p.narrow;
  f.w1 = c.wop[0];
  f.w2 = c.wop[1];
  f.w3 = c.wop[2];
  const double ffl = (apply_too ? 4.0 : 0.0) * p.BH * n * dh + 6.0 * p.BH * n * dh;
  int rc = timed(LACT_KCLASS_FWD, ffl, c.s, [&] { return launch_fwd(f, p.bf16, c.s); });
  if (rc) return rc;

  BwdArgs b{};
  int nb = 0;
  const bool fused = p.fused;
  if (fused) {
    // gradient and update of whole rows (with the momentum state when there
    // is one); the new bf16 copies go to the other set
    BwdSeg& g = b.seg[nb++];
    const int rt = grad_upd_tile().rows;
    g.kind = BWD_GRAD_UPD;
    g.tiles_m = (int)(2 * cdiv(p.h, rt) + cdiv(p.d, rt));
    g.tiles_n = 1;
    g.nsplit = 1;
    g.nblocks = p.BH * g.tiles_m;
    g.rows = n;
    g.split_len = n;
    g.a0 = op(c.ws + p.off_upd[1], p.h, p.C * p.h);   // eta dz1
    g.a1 = op(c.ws + p.off_upd[2], p.h, p.C * p.h);   // eta dz3
    g.b0 = op(c.k + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);
    g.a2 = op(c.v + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);
    g.b1 = op(c.ws + p.off_upd[0], p.h, p.C * p.h);   // eta hidden
    for (int m = 0; m < 3; ++m) {
      g.W[m] = c.W[m];
      g.Wb[m] = c.wb[c.wset ^ 1][m];
    }
    if (c.beta) {
      for (int m = 0; m < 3; ++m) g.M[m] = c.M[m];
      g.bbar = bbar_of(c);
      g.bbar_stride = kBetaBatch;
    }
  }
  // Otherwise the gradient contractions, split over tokens (a split past the
  // chunk's end writes zeros so the update always sums p.nsplit partials),
  // and the update in a launch of its own (finish_update).
  const TileShape g13 = bwd_tile(BWD_GRAD13, p.bf16, p.narrow), g2 = bwd_tile(BWD_GRAD2, p.bf16, p.narrow);
  if (!fused) {   // W1's and W3's gradients
    BwdSeg& g = b.seg[nb++];
    g.kind = BWD_GRAD13;
    g.tiles_m = (int)cdiv(p.h, g13.rows);
    g.tiles_n = (int)cdiv(p.d, g13.cols);
    g.nsplit = p.nsplit;
    g.nblocks = p.BH * g.tiles_m * g.tiles_n * p.nsplit;
    g.rows = n;
    g.split_len = p.split_len;
    g.a0 = op(c.ws + p.off_upd[1], p.h, p.C * p.h);   // eta dz1
    g.a1 = op(c.ws + p.off_upd[2], p.h, p.C * p.h);   // eta dz3
    g.b0 = op(c.k + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);
    g.out = c.ws + p.off_step;
    g.out_inst = 3 * dh;
    g.out_split = (int64_t)p.BH * 3 * dh;
    set_tile_sums(c, g, 0);
  }
  if (!fused) {   // W2's gradient
    BwdSeg& g = b.seg[nb++];
    g.kind = BWD_GRAD2;
    g.tiles_m = (int)cdiv(p.d, g2.rows);
    g.tiles_n = (int)cdiv(p.h, g2.cols);
    g.nsplit = p.nsplit;
    g.nblocks = p.BH * g.tiles_m * g.tiles_n * p.nsplit;
    g.rows = n;
    g.split_len = p.split_len;
    g.a0 = op(c.v + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);
    g.b0 = op(c.ws + p.off_upd[0], p.h, p.C * p.h);   // eta hidden
    g.out = c.ws + p.off_step;
    g.out_inst = 3 * dh;
    g.out_split = (int64_t)p.BH * 3 * dh;
    g.out_off = dh;   // W2's partials follow W1's
    set_tile_sums(c, g, 1);
  }
  if (apply_too) {
    // with ns_out the output tiles wait for the Newton-Schulz launch, which
    // follows this one (finish_update) and still reads this copy set's W2
    BwdArgs& ob = c.out_pending;
    BwdSeg& o = p.ns_out ? ob.seg[0] : b.seg[nb++];
    o = BwdSeg{};
    o.kind = BWD_OUT;
    o.tiles_m = (int)cdiv(p.d, bwd_tile(BWD_OUT, p.bf16, p.narrow).rows);
    o.tiles_n = (int)cdiv(n, bwd_tile(BWD_OUT, p.bf16, p.narrow).cols);
    o.nsplit = 1;
    o.nblocks = p.BH * o.tiles_m * o.tiles_n;
    o.rows = n;
    o.a0 = op(c.ws + p.off_hq, p.h, p.cap * p.h);
    o.b0 = c.wop[1];
    o.out = c.o + s0 * p.d * p.esz;
    o.out_inst = c.dsc->n_q * p.d;
    if (p.ns_out) {
      ob.nseg = 1;
      ob.total_blocks = o.nblocks;
      ob.d = p.d;
      ob.h = p.h;
      ob.narrow = p.narrow;
      c.out_flops = 2.0 * p.BH * n * dh;
      c.has_out = true;
    }
  }
  b.nseg = nb;
  b.total_blocks = 0;
  for (int i = 0; i < nb; ++i) b.total_blocks += b.seg[i].nblocks;
  b.d = p.d;
  b.h = p.h;
  b.narrow = p.narrow;
  const double bfl = (apply_too && !p.ns_out ? 2.0 : 0.0) * p.BH * n * dh + 6.0 * p.BH * n * dh;
  rc = timed(LACT_KCLASS_BWD, bfl, c.s, [&] { return launch_bwd(b, p.bf16, c.s); });
  if (rc) return rc;
  if (fused) {   // the update is done; the next launches read the new copies
    use_wset(c, c.wset ^ 1);
    return LACT_OK;
  }
  if (c.grad_only) return LACT_OK;
  return finish_update(c);
}

// The gradient partials are in place: Newton-Schulz (Muon) and the weight
// update with its row normalisation and the operand copies.
int finish_update(Ctx& c) {
  const Plan& p = c.p;
  const int64_t dh = (int64_t)p.d * p.h;
  int rc = LACT_OK;
  UpdArgs u{};
  for (int m = 0; m < p.nmat; ++m) {
    u.W[m] = c.W[m];
    u.Wsrc[m] = c.Wsrc[m];
    u.Wb[m] = p.bf16 ? c.wb[c.wset][m] : nullptr;
  }
  u.nmat = p.nmat;
  if (p.muon) {
    c.ns_updated = false;
    rc = newton_schulz(c);
    if (rc) return rc;
    if (c.ns_updated) return LACT_OK;
    u.step = reinterpret_cast<const float*>(c.ws + p.off_y32);
    u.nsplit = 1;
    u.step_split = 0;
  } else {
    u.step = reinterpret_cast<const float*>(c.ws + p.off_step);
    u.nsplit = p.nsplit;
    u.step_split = (int64_t)p.BH * p.nmat * dh;
    if (c.beta) {   // with Muon the state was advanced before Newton-Schulz
      for (int j = 0; j < p.nmat; ++j) u.M[j] = c.M[j];
      u.bbar = bbar_of(c);
      u.bbar_stride = kBetaBatch;
    }
  }
  u.BH = p.BH;
  u.d = p.d;
  u.h = p.h;
  u.rows_total = p.BH * (p.linear ? p.d : 2 * p.h + p.d);
  return timed(LACT_KCLASS_UPDATE, 0.0, c.s, [&] { return launch_update(u, p.bf16, c.s); });
}

// Linear fast weight f_W(x) = W x (W: d x d): the gradient partials
// P = sum_i v_i (eta_i k_i)^T (= -g) of key rows [s0, s1) from eta k and V in
// one GRAD2 contraction, with the apply o = W q of the same rows in the same
// launch when apply_too.
int update_chunk_linear(Ctx& c, int64_t s0, int64_t s1, bool apply_too) {
  const Plan& p = c.p;
  const int64_t n = s1 - s0;
  const int64_t dd = (int64_t)p.d * p.d;
  int rc = timed(LACT_KCLASS_FWD, 0.0, c.s, [&] {
    return launch_scale_rows(c.k + s0 * p.d * p.esz, c.eta + s0, c.ws + p.off_upd[0], p.BH, n, p.d,
                             c.dsc->n_kv * p.d, c.dsc->n_kv, p.C * p.d, p.bf16, c.s);
  });
  if (rc) return rc;
  BwdArgs b{};
  int nb = 0;
  const TileShape g2 = bwd_tile(BWD_GRAD2, p.bf16, p.narrow);
  {
    BwdSeg& g = b.seg[nb++];
    g.kind = BWD_GRAD2;
    g.tiles_m = (int)cdiv(p.d, g2.rows);
    g.tiles_n = (int)cdiv(p.d, g2.cols);
    g.nsplit = p.nsplit;
    g.nblocks = p.BH * g.tiles_m * g.tiles_n * p.nsplit;
    g.rows = n;
    g.split_len = p.split_len;
    g.a0 = op(c.v + s0 * p.d * p.esz, p.d, c.dsc->n_kv * p.d);   // V
    g.b0 = op(c.ws + p.off_upd[0], p.d, p.C * p.d);               // eta K
    g.out = c.ws + p.off_step;
    g.out_inst = dd;
    g.out_split = (int64_t)p.BH * dd;
    g.out_off = 0;
    set_tile_sums(c, g, 0);
  }
  if (apply_too) {
    BwdSeg& o = b.seg[nb++];
    o.kind = BWD_OUT;
    o.tiles_m = (int)cdiv(p.d, bwd_tile(BWD_OUT, p.bf16, p.narrow).rows);
    o.tiles_n = (int)cdiv(n, bwd_tile(BWD_OUT, p.bf16, p.narrow).cols);
    o.nsplit = 1;
    o.nblocks = p.BH * o.tiles_m * o.tiles_n;
    o.rows = n;
    o.a0 = op(c.q + s0 * p.d * p.esz, p.d, c.dsc->n_q * p.d);
    o.b0 = c.wop[0];
    o.out = c.o + s0 * p.d * p.esz;
    o.out_inst = c.dsc->n_q * p.d;
  }
  b.nseg = nb;
  b.total_blocks = 0;
  for (int i = 0; i < nb; ++i) b.total_blocks += b.seg[i].nblocks;
  b.d = p.d;
  b.h = p.d;   // OUT contracts over d; GRAD2's columns run over d
  b.narrow = p.narrow;
  const double bfl = (apply_too ? 2.0 : 0.0) * p.BH * n * dd + 2.0 * p.BH * n * dd;
  rc = timed(LACT_KCLASS_BWD, bfl, c.s, [&] { return launch_bwd(b, p.bf16, c.s); });
  if (rc) return rc;
  return finish_update(c);
}

// Validation and context of every entry point (no HIP call); beta == nullptr
// and M == nullptr: plain updates; M: momentum with state M (beta required
// when there are key tokens).
int setup(Ctx& c, const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
          const float* beta, float* W1, float* W2, float* W3, float* const M[3], void* o, void* workspace,
          size_t workspace_bytes, void* stream, bool use_scratch = false) {
  int rc = check_desc(desc);
  if (rc) return rc;
  const bool any_kv = desc->n_kv > 0, any_q = desc->n_q > 0;
  const bool linear = desc->fast_weight == LACT_FW_LINEAR;   // W2, W3 (M2, M3) unused
  if (!W1 || (!linear && (!W2 || !W3))) return LACT_EINVAL;
  if (any_q && (!q || !o)) return LACT_EINVAL;
  if (any_kv && (!k || !v || !eta)) return LACT_EINVAL;
  if (M && (!M[0] || (!linear && (!M[1] || !M[2])) || (any_kv && !beta))) return LACT_EINVAL;
  if (misaligned(W1) || (!linear && (misaligned(W2) || misaligned(W3)))) return LACT_EALIGN;
  if (any_q && (misaligned(q) || misaligned(o))) return LACT_EALIGN;
  if (any_kv && (misaligned(k) || misaligned(v) || ((uintptr_t)eta & 3))) return LACT_EALIGN;
  if (M && (misaligned(M[0]) || (!linear && (misaligned(M[1]) || misaligned(M[2]))))) return LACT_EALIGN;
  if (M && any_kv && ((uintptr_t)beta & 3)) return LACT_EALIGN;
  c = Ctx{};
  c.dsc = desc;
  c.p = make_plan(desc);
  if (use_scratch) {   // the fixed per-device array; its address is resolved by the caller
    if (c.p.total > LACT_NOALLOC_SCRATCH_BYTES) return LACT_ESCRATCH;
  } else {
    if (!workspace || workspace_bytes < c.p.total) return LACT_EWORKSPACE;
    if ((uintptr_t)workspace & (kAlign - 1)) return LACT_EALIGN;
  }
  c.q = (const uint8_t*)q;
  c.k = (const uint8_t*)k;
  c.v = (const uint8_t*)v;
  c.eta = eta;
  c.W[0] = W1;
  c.W[1] = W2;
  c.W[2] = W3;
  c.o = (uint8_t*)o;
  c.ws = (uint8_t*)workspace;
  c.s = (hipStream_t)stream;
  if (M) {
    c.beta = beta;
    for (int j = 0; j < 3; ++j) c.M[j] = M[j];
  }
  return LACT_OK;
}

// Operand copies of the initial fast weights (bf16 I/O) or the fp32 state.
int prepare_weights(Ctx& c) {
  const Plan& p = c.p;
  const int64_t dh = (int64_t)p.d * p.h;
  if (p.bf16) {
    const float* Wf[3] = {c.W[0], p.linear ? nullptr : c.W[1], p.linear ? nullptr : c.W[2]};
    for (int m = 0; m < 3; ++m) {
      c.wb[0][m] = c.ws + p.off_wb[m];
      c.wb[1][m] = c.ws + p.off_wb2[m];
    }
    const int rc =
        timed(LACT_KCLASS_PREP, 0.0, c.s, [&] { return launch_prep(Wf, c.wb[0], p.BH, p.d, p.h, c.s); });
    if (rc) return rc;
    use_wset(c, 0);
  } else {
    c.wop[0] = op(c.W[0], p.d, dh);
    c.wop[1] = op(c.W[1], p.h, dh);
    c.wop[2] = op(c.W[2], p.d, dh);
  }
  return LACT_OK;
}

// Momentum factors of `nchunks` chunks of `len` tokens from token t0 (the
// last bounded by `end`) into slots 0.. of the chunk-mean section.
int beta_means(Ctx& c, int64_t t0, int64_t len, int64_t end, int nchunks) {
  BetaArgs ba{};
  ba.beta = c.beta;
  ba.n_kv = c.dsc->n_kv;
  ba.chunk = len;
  ba.t0 = t0;
  ba.end = end;
  ba.nchunks = nchunks;
  ba.BH = c.p.BH;
  ba.bbar = reinterpret_cast<float*>(c.ws + c.p.off_bbar);
  ba.stride = kBetaBatch;
  return timed(LACT_KCLASS_UPDATE, 0.0, c.s, [&] { return launch_beta_mean(ba, c.s); });
}

// Device address of `scratch` on the device that stream `s` belongs to (the
// current device for the null stream): looked up once per device, with that
// device current, and kept for the life of the process.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch[kMaxDevices] = {};

int scratch_for_stream(hipStream_t s, uint8_t** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return record_hip(e);
  int dev = cur;
  if (s) {
    hipDevice_t sd = 0;
    if ((e = hipStreamGetDevice(s, &sd)) != hipSuccess) return record_hip(e);
    dev = (int)sd;
  }
  if (dev < 0 || dev >= kMaxDevices) return LACT_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return record_hip(e);
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t back = hipSetDevice(cur);
      if (e == hipSuccess) e = back;
    }
    if (e != hipSuccess) return record_hip(e);
    if (!p || ((uintptr_t)p & (kAlign - 1))) {
      snprintf(g_hip_err, sizeof g_hip_err, "scratch array at %p: not 256-byte aligned", p);
      return LACT_EHIP;
    }
    g_scratch[dev] = reinterpret_cast<uint8_t*>(p);
  }
  *out = g_scratch[dev];
  return LACT_OK;
}

// lact_forward and lact_forward_momentum: uniform chunks of desc->chunk tokens
// in desc->order, then the apply-only tail. With use_scratch the workspace is
// the device's scratch array (lact_forward_noalloc).
int run_forward(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                const float* beta, float* W1, float* W2, float* W3, float* const M[3], void* o,
                void* workspace, size_t workspace_bytes, void* stream, bool use_scratch = false) {
  Ctx c;
  int rc = setup(c, desc, q, k, v, eta, beta, W1, W2, W3, M, o, workspace, workspace_bytes, stream, use_scratch);
  if (rc) return rc;
  if (use_scratch) {
    rc = scratch_for_stream(c.s, &c.ws);
    if (rc) return rc;
  }
  rc = prepare_weights(c);
  if (rc) return rc;
  const int64_t n_kv = desc->n_kv, n_q = desc->n_q, C = desc->chunk;
  const int64_t nchunks = cdiv(n_kv, C);
  for (int64_t s0 = 0; s0 < n_kv; s0 += C) {
    const int64_t s1 = std::min(n_kv, s0 + C);
    c.chunk_idx = s0 / C;
    if (c.beta && c.chunk_idx % kBetaBatch == 0) {
      rc = beta_means(c, s0, C, n_kv, (int)std::min<int64_t>(kBetaBatch, nchunks - c.chunk_idx));
      if (rc) return rc;
    }
    if (desc->order == LACT_APPLY_THEN_UPDATE) {
      rc = update_chunk(c, s0, s1, true);
    } else {
      rc = update_chunk(c, s0, s1, false);
      if (!rc) rc = apply_rows(c, s0, s1 == n_kv ? n_q : s1);
    }
    if (rc) return rc;
  }
  if (desc->order == LACT_APPLY_THEN_UPDATE || n_kv == 0) rc = apply_rows(c, n_kv, n_q);
  return rc;
}

bool is_update(int mode) { return mode != LACT_SEG_APPLY_ONLY; }
bool is_apply(int mode) { return mode != LACT_SEG_UPDATE_ONLY; }

int check_segments(const lact_desc* desc, const lact_segment* segs, int64_t nseg) {
  if (nseg < 0 || (nseg > 0 && !segs)) return LACT_EINVAL;
  for (int64_t i = 0; i < nseg; ++i) {
    const lact_segment& g = segs[i];
    if (g.mode < LACT_SEG_APPLY_THEN_UPDATE || g.mode > LACT_SEG_APPLY_ONLY || g.reserved != 0) return LACT_EINVAL;
    if (g.begin < 0 || g.end <= g.begin) return LACT_EINVAL;
    if (is_update(g.mode) && (g.end > desc->n_kv || g.end - g.begin > desc->chunk)) return LACT_EINVAL;
    if (is_apply(g.mode) && g.end > desc->n_q) return LACT_EINVAL;
  }
  return LACT_OK;
}

// lact_forward_schedule: caller-given segments; rows that no apply segment
// covers are zeroed first.
int run_schedule(const lact_desc* desc, const lact_segment* segs, int64_t nseg, const void* q, const void* k,
                 const void* v, const float* eta, const float* beta, float* W1, float* W2, float* W3,
                 float* const M[3], void* o, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  rc = check_segments(desc, segs, nseg);
  if (rc) return rc;
  Ctx c;
  rc = setup(c, desc, q, k, v, eta, beta, W1, W2, W3, M, o, workspace, workspace_bytes, stream);
  if (rc) return rc;
  const Plan& p = c.p;
  std::vector<std::pair<int64_t, int64_t>> cover;
  for (int64_t i = 0; i < nseg; ++i)
    if (is_apply(segs[i].mode)) cover.emplace_back(segs[i].begin, segs[i].end);
  std::sort(cover.begin(), cover.end());
  int64_t at = 0;
  const int64_t row_bytes = (int64_t)p.d * p.esz;
  for (size_t i = 0; i <= cover.size(); ++i) {
    const int64_t b = i < cover.size() ? cover[i].first : desc->n_q;
    if (b > at) {
      const int64_t e = b;
      rc = timed(LACT_KCLASS_PREP, 0.0, c.s,
                 [&] { return launch_zero_rows(c.o, p.BH, row_bytes, desc->n_q, at, e, c.s); });
      if (rc) return rc;
    }
    if (i < cover.size()) at = std::max(at, cover[i].second);
  }
  rc = prepare_weights(c);
  if (rc) return rc;
  c.chunk_idx = 0;
  for (int64_t i = 0; i < nseg; ++i) {
    const lact_segment& g = segs[i];
    if (c.beta && is_update(g.mode)) {
      rc = beta_means(c, g.begin, g.end - g.begin, g.end, 1);
      if (rc) return rc;
    }
    switch (g.mode) {
      case LACT_SEG_APPLY_THEN_UPDATE:
        rc = update_chunk(c, g.begin, g.end, true);
        break;
      case LACT_SEG_UPDATE_THEN_APPLY:
        rc = update_chunk(c, g.begin, g.end, false);
        if (!rc) rc = apply_rows(c, g.begin, g.end);
        break;
      case LACT_SEG_UPDATE_ONLY:
        rc = update_chunk(c, g.begin, g.end, false);
        break;
      default:
        rc = apply_rows(c, g.begin, g.end);
    }
    if (rc) return rc;
  }
  return LACT_OK;
}

// ---------------------------------------------------------------- backward of Newton-Schulz
// Muon's step of a chunk (App. A, Details of Muon; §3.2) and its reverse, on
// slots s = inst * nmat + j of wide [m x n] fp32 matrices (a stored matrix
// with more rows than columns is transposed into its slot). The reverse
// replays the iteration from the chunk's gradient, keeping the fp16 operand
// copies of every iterate X_k, of A_k = X_k X_k^T and of B_k = b A_k + c A_k^2,
// and then goes back one step at a time:
//   dB = dX' X^T,  S = dB + dB^T,  M = b S + c (S A + (S A)^T)  (= dA + dA^T),
//   dX = a dX' + B dX' + M X,
// and through the scaling X_0 = G / (||G|| + eps). Products: the k_bwd kinds
// (OUT for sums along rows, GRAD2 for sums down columns, fp32 partials) on
// fp16 operand copies with bf16 I/O, fp32 ones with fp32 I/O; fp32 iterates.
struct NsBwdLayout {
  int S, m, n;
  int64_t iters;   // slices of the iterates and steps: 1 (replayed per chunk) or one per chunk (kept)
  int es;          // bytes per operand element: 2 (fp16) or 4 (fp32, with fp32 I/O)
  size_t g, x32, p1, p2, xo, ao, bo, to, qo, so, mo, dbo, nrm, dot, dotp, pstep, ustep, ug, total;
};

// Chunks whose Newton-Schulz iterates and steps the backward keeps (each
// chunk's iteration then runs once, in the replay), within this many bytes.
constexpr double kKeepIterBytes = 24.0 * (1 << 30);

size_t ns_bwd_layout(const Plan& p, int steps, size_t o, NsBwdLayout* N, int64_t nch = 1) {
  N->S = p.BH * p.nmat;
  N->m = std::min(p.d, p.h);
  N->n = std::max(p.d, p.h);
  const size_t mn = (size_t)N->m * N->n, mm = (size_t)N->m * N->m, S = N->S;
  N->es = p.bf16 ? 2 : 4;
  const size_t es = (size_t)N->es;
  const double per = ((double)std::max(steps, 1) * S * (mn + 2 * mm) * es + (double)S * mn * 4.0);
  N->iters = nch > 1 && per * nch <= kKeepIterBytes ? nch : 1;
  const size_t it = (size_t)N->iters;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  N->g = take(S * mn * 4);
  N->x32 = take(S * mn * 4);
  N->p1 = take(S * mn * 4);
  N->p2 = take(S * mn * 4);
  N->xo = take(it * std::max(steps, 1) * S * mn * es);
  N->ao = take(it * std::max(steps, 1) * S * mm * es);
  N->bo = take(it * std::max(steps, 1) * S * mm * es);
  N->to = take(S * mn * es);
  N->qo = take(S * mm * es);
  N->so = take(S * mm * es);
  N->mo = take(S * mm * es);
  N->dbo = take(S * mm * es);
  N->nrm = take(S * 4);
  N->dot = take(S * 4);
  N->dotp = take(S * 32 * 4);   // the dot products' per-workgroup partials
  N->pstep = take(it * S * mn * 4);   // stored layouts [inst][nmat][d h]
  N->ustep = take(S * mn * 4);
  N->ug = take(S * mn * 4);
  N->total = o;
  return o;
}

struct NsBwd {
  const Plan& p;
  const NsBwdLayout& N;
  uint8_t* ws;
  hipStream_t s;
  int steps;
  int R[3], L[3];   // stored shape of matrix j
  int64_t ci = 0;   // the chunk whose slice of kept iterates is used (with one slice: always slice 0)
  template <class T>
  T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
  int64_t mn() const { return (int64_t)N.m * N.n; }
  int64_t mm() const { return (int64_t)N.m * N.m; }
  bool tall(int j) const { return R[j] > L[j]; }

  // stored [inst][nmat][R x L] (nsum splits `split` apart, times sign) <-> wide slots
  int gather(const float* src, int nsum, int64_t split, float sign, float* wide) const {
    CopySeg cs[3] = {};
    const int64_t dh = (int64_t)p.d * p.h;
    for (int j = 0; j < p.nmat; ++j) {
      CopySeg& c = cs[j];
      c.W = src + j * dh;
      c.w_inst = p.nmat * dh;
      c.R = R[j];
      c.L = L[j];
      c.nsum = nsum;
      c.split = split;
      c.sign = sign;
      if (tall(j)) {
        c.dstT = wide + j * mn();
        c.ldT = R[j];
        c.dstT_inst = p.nmat * mn();
      } else {
        c.dst = wide + j * mn();
        c.ld = L[j];
        c.dst_inst = p.nmat * mn();
      }
    }
    return timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_copies_f32(cs, p.nmat, p.BH, s); });
  }
  // the same from per-matrix slabs ([BH][R x L] each)
  int gather_slabs(const float* const src[3], float sign, float* wide) const {
    CopySeg cs[3] = {};
    for (int j = 0; j < p.nmat; ++j) {
      CopySeg& c = cs[j];
      c.W = src[j];
      c.w_inst = (int64_t)R[j] * L[j];
      c.R = R[j];
      c.L = L[j];
      c.sign = sign;
      if (tall(j)) {
        c.dstT = wide + j * mn();
        c.ldT = R[j];
        c.dstT_inst = p.nmat * mn();
      } else {
        c.dst = wide + j * mn();
        c.ld = L[j];
        c.dst_inst = p.nmat * mn();
      }
    }
    return timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_copies_f32(cs, p.nmat, p.BH, s); });
  }
  int scatter(const float* wide, float sign, float* dst) const {
    CopySeg cs[3] = {};
    const int64_t dh = (int64_t)p.d * p.h;
    for (int j = 0; j < p.nmat; ++j) {
      CopySeg& c = cs[j];
      c.W = wide + j * mn();
      c.w_inst = p.nmat * mn();
      c.R = N.m;
      c.L = N.n;
      c.sign = sign;
      if (tall(j)) {   // the stored matrix is the slot's transpose
        c.dstT = dst + j * dh;
        c.ldT = L[j];
        c.dstT_inst = p.nmat * dh;
      } else {
        c.dst = dst + j * dh;
        c.ld = L[j];
        c.dst_inst = p.nmat * dh;
      }
    }
    return timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_copies_f32(cs, p.nmat, p.BH, s); });
  }
  // out[i][j] = sum_e a[i][e] b[j][e] over K per slot (rows of a: `rows`, of b: rows_out)
  int out(const void* a, int64_t a_ld, int64_t a_inst, const void* b, int64_t b_ld, int64_t b_inst,
          void* o, int rows, int rows_out, int K) const {
    BwdArgs x{};
    const TileShape t = bwd_tile(BWD_OUT, !f32(), false);
    BwdSeg& g = x.seg[0];
    g.kind = BWD_OUT;
    g.tiles_m = (int)cdiv(rows_out, t.rows);
    g.tiles_n = (int)cdiv(rows, t.cols);
    g.nsplit = 1;
    g.nblocks = N.S * g.tiles_m * g.tiles_n;
    g.rows = rows;
    g.a0 = op(a, a_ld, a_inst);
    g.b0 = op(b, b_ld, b_inst);
    g.out = o;
    g.out_inst = (int64_t)rows * rows_out;
    g.klen = K;
    x.nseg = 1;
    x.total_blocks = g.nblocks;
    x.d = rows_out;
    x.h = K;
    x.narrow = 0;
    return timed(LACT_KCLASS_NS, 2.0 * N.S * rows * rows_out * K, s,
                 [&] { return f32() ? launch_bwd(x, false, s) : launch_bwd_f16(x, s); });
  }
  // out = a^T b per slot: a [m x m] (rows i), b [m x n] (rows i), fp32 [m x n]; up to two at once
  int grad2(const void* const* a, const void* const* b, float* const* o, int nseg) const {
    BwdArgs x{};
    // fp16: 128 x 256 tiles (the narrow kinds), twice the workgroups of the
    // 256 x 256 ones, so that the slots' tiles fill the chip
    const bool half = !f32();
    const TileShape t = bwd_tile(BWD_GRAD2, !f32(), half);
    for (int i = 0; i < nseg; ++i) {
      BwdSeg& g = x.seg[i];
      g.kind = BWD_GRAD2;
      g.tiles_m = (int)cdiv(N.m, t.rows);
      g.tiles_n = (int)cdiv(N.n, t.cols);
      g.nsplit = 1;
      g.nblocks = N.S * g.tiles_m * g.tiles_n;
      g.rows = N.m;
      g.split_len = cdiv(N.m, 32) * 32;
      g.a0 = op(a[i], N.m, mm());
      g.b0 = op(b[i], N.n, mn());
      g.out = o[i];
      g.out_inst = mn();
      g.out_split = N.S * mn();
      g.out_off = 0;
    }
    x.nseg = nseg;
    x.total_blocks = 0;
    for (int i = 0; i < nseg; ++i) x.total_blocks += x.seg[i].nblocks;
    x.d = N.m;
    x.h = N.n;
    x.narrow = half ? 1 : 0;
    return timed(LACT_KCLASS_NS, 2.0 * nseg * N.S * mm() * N.n, s,
                 [&] { return f32() ? launch_bwd(x, false, s) : launch_bwd_f16(x, s); });
  }
  int lin(int mode, const float* x, const float* y, const float* p1, const float* p2, const float* sc,
          const float* sc2, float a, float* o32, void* oc) const {
    NsLinArgs l{};
    l.mode = mode;
    l.x = x;
    l.y = y;
    l.p1 = p1;
    l.p2 = p2;
    l.sc = sc;
    l.sc2 = sc2;
    l.a = a;
    l.eps = (float)kNsEps;
    l.out32 = o32;
    if (f32()) l.outc32 = reinterpret_cast<float*>(oc);   // the operand copy: fp32 with fp32 I/O, else fp16
    else l.out16 = reinterpret_cast<_Float16*>(oc);
    l.S = N.S;
    l.len = mn();
    return timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_ns_lin(l, s); });
  }
  size_t sk(int k) const { return (size_t)(ci % N.iters) * steps + k; }   // step k of this chunk's slice
  bool f32() const { return N.es == 4; }   // fp32 operands (fp32 I/O), else fp16
  uint8_t* Xo(int k) const { return at<uint8_t>(N.xo) + sk(k) * N.S * mn() * N.es; }
  uint8_t* Ao(int k) const { return at<uint8_t>(N.ao) + sk(k) * N.S * mm() * N.es; }
  uint8_t* Bo(int k) const { return at<uint8_t>(N.bo) + sk(k) * N.S * mm() * N.es; }
  uint8_t* buf(size_t off) const { return at<uint8_t>(off); }
  // out = alpha X + beta (Y + Y^T) per [m x m] slot in the operand type (X may be nullptr)
  int sym(const void* X, float alpha, const void* Y, float beta, void* o) const {
    return timed(LACT_KCLASS_NS, 0.0, s, [&] {
      return f32() ? launch_sym32(reinterpret_cast<const float*>(X), alpha, reinterpret_cast<const float*>(Y), beta,
                                  reinterpret_cast<float*>(o), N.S, N.m, s)
                   : launch_sym(reinterpret_cast<const _Float16*>(X), alpha, reinterpret_cast<const _Float16*>(Y),
                                beta, reinterpret_cast<_Float16*>(o), N.S, N.m, s);
    });
  }
  float* pst() const { return at<float>(N.pstep) + (size_t)(ci % N.iters) * N.S * mn(); }   // the step, negated
  bool kept() const { return N.iters > 1; }

  // What the reverse needs besides the kept iterates: the iteration's input
  // G (from P or the slabs, as forward) and its squared norm.
  int prepare(const float* P, int nsplit, int64_t split, const float* const* slabs = nullptr) const {
    float* G = at<float>(N.g);
    int rc = slabs ? gather_slabs(slabs, 1.0f, G) : gather(P, nsplit, split, -1.0f, G);
    if (!rc) rc = timed(LACT_KCLASS_NS, 0.0, s, [&] {
      return launch_slot_dot(G, G, N.S, mn(), at<float>(N.nrm), at<float>(N.dotp), s);
    });
    return rc;
  }
  // The step -Muon(g) of the gradient whose negated split partials are
  // P (stored layout), into pstep (stored layout, one split); with slabs,
  // of the momentum state in per-matrix slabs instead.
  int forward(const float* P, int nsplit, int64_t split, const float* const* slabs = nullptr) const {
    float* G = at<float>(N.g);
    float* X = at<float>(N.x32);
    int rc = slabs ? gather_slabs(slabs, 1.0f, G) : gather(P, nsplit, split, -1.0f, G);
    if (!rc) rc = timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_slot_dot(G, G, N.S, mn(), at<float>(N.nrm), at<float>(N.dotp), s); });
    if (!rc) rc = lin(0, G, nullptr, nullptr, nullptr, at<float>(N.nrm), nullptr, 0.f, X, steps > 0 ? Xo(0) : nullptr);
    for (int k = 0; k < steps && !rc; ++k) {
      rc = out(Xo(k), N.n, mn(), Xo(k), N.n, mn(), Ao(k), N.m, N.m, N.n);   // A = X X^T
      if (!rc) rc = out(Ao(k), N.m, mm(), Ao(k), N.m, mm(), buf(N.qo), N.m, N.m, N.m);   // A A
      if (!rc) rc = sym(Ao(k), (float)kNsB, buf(N.qo), 0.5f * (float)kNsC, Bo(k));   // B = b A + c A A (symmetrised)
      const void* a2[1] = {Bo(k)};
      const void* b2[1] = {Xo(k)};
      float* o2[1] = {at<float>(N.p1)};
      if (!rc) rc = grad2(a2, b2, o2, 1);   // B X
      if (!rc) rc = lin(1, X, nullptr, at<float>(N.p1), nullptr, nullptr, nullptr, (float)kNsA, X,
                        k + 1 < steps ? Xo(k + 1) : nullptr);
    }
    if (!rc) rc = scatter(X, -1.0f, pst());
    return rc;
  }
  // From the update's cotangent of U = W - step (ustep, stored layout), the
  // gradient's cotangent negated (-dg, stored layout) into ug.
  int reverse() const {
    float* G = at<float>(N.g);
    float* X = at<float>(N.x32);
    uint8_t* T = buf(N.to);
    int rc = gather(at<float>(N.ustep), 1, 0, -1.0f, X);   // d step = -dU
    if (!rc) rc = lin(1, X, nullptr, nullptr, nullptr, nullptr, nullptr, 1.0f, nullptr, T);
    for (int k = steps - 1; k >= 0 && !rc; --k) {
      rc = out(T, N.n, mn(), Xo(k), N.n, mn(), buf(N.dbo), N.m, N.m, N.n);   // dB = dX' X^T
      if (!rc) rc = sym(nullptr, 0.f, buf(N.dbo), 1.0f, buf(N.so));
      if (!rc) rc = out(buf(N.so), N.m, mm(), Ao(k), N.m, mm(), buf(N.qo), N.m, N.m, N.m);
      if (!rc) rc = sym(buf(N.so), (float)kNsB, buf(N.qo), (float)kNsC, buf(N.mo));   // M = b S + c (S A + (S A)^T)
      const void* a2[2] = {Bo(k), buf(N.mo)};
      const void* b2[2] = {T, Xo(k)};
      float* o2[2] = {at<float>(N.p1), at<float>(N.p2)};
      if (!rc) rc = grad2(a2, b2, o2, 2);   // B dX', M X
      if (!rc) rc = lin(1, X, nullptr, at<float>(N.p1), at<float>(N.p2), nullptr, nullptr, (float)kNsA, X,
                        k > 0 ? T : nullptr);
    }
    if (!rc) rc = timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_slot_dot(X, G, N.S, mn(), at<float>(N.dot), at<float>(N.dotp), s); });
    if (!rc) rc = lin(2, X, G, nullptr, nullptr, at<float>(N.nrm), at<float>(N.dot), 0.f, X, nullptr);
    if (!rc) rc = scatter(X, -1.0f, at<float>(N.ug));
    return rc;
  }
};

// One segment of the backward's schedule: a LACT_SEG_* mode over tokens
// [b, e) and the number of updates before it: an update segment's own index
// among the updates, and the index of the weight that an apply before its
// update, or an apply-only segment, uses.
struct BSeg {
  int mode;
  int64_t b, e;
  int64_t before;
};

// The uniform schedule of lact_forward (chunks of desc->chunk, then the
// apply-only tail), or the caller's segments checked for the backward: the
// update ranges must not overlap each other, nor the apply ranges (the
// reverse writes the cotangents of a token's rows once).
int backward_segments(const lact_desc* desc, const lact_segment* segs, int64_t nseg, std::vector<BSeg>* out,
                      int64_t* nupd, int64_t* longest_apply) {
  out->clear();
  *nupd = 0;
  *longest_apply = 0;
  if (nseg < 0) {
    const int mode = desc->order == LACT_UPDATE_THEN_APPLY ? LACT_SEG_UPDATE_THEN_APPLY : LACT_SEG_APPLY_THEN_UPDATE;
    for (int64_t s0 = 0; s0 < desc->n_kv; s0 += desc->chunk)
      out->push_back(BSeg{mode, s0, std::min(desc->n_kv, s0 + desc->chunk), (*nupd)++});
    if (desc->n_q > desc->n_kv) {
      out->push_back(BSeg{LACT_SEG_APPLY_ONLY, desc->n_kv, desc->n_q, *nupd});
      *longest_apply = desc->n_q - desc->n_kv;
    }
    return LACT_OK;
  }
  int rc = check_segments(desc, segs, nseg);
  if (rc) return rc;
  std::vector<std::pair<int64_t, int64_t>> ur, ar;
  for (int64_t i = 0; i < nseg; ++i) {
    const lact_segment& g = segs[i];
    out->push_back(BSeg{g.mode, g.begin, g.end, *nupd});
    if (is_update(g.mode)) {
      ur.emplace_back(g.begin, g.end);
      ++*nupd;
    }
    if (is_apply(g.mode)) ar.emplace_back(g.begin, g.end);
    if (g.mode == LACT_SEG_APPLY_ONLY) *longest_apply = std::max(*longest_apply, g.end - g.begin);
  }
  for (auto* r : {&ur, &ar}) {
    std::sort(r->begin(), r->end());
    for (size_t i = 1; i < r->size(); ++i)
      if ((*r)[i].first < (*r)[i - 1].second) return LACT_EUNSUPPORTED;
  }
  return LACT_OK;
}

// Zeroes rows [r0, r1) of every instance of a per-token fp32 array of `cols`
// values per row ([BH][rows][cols]).
int zero_f32_rows(float* x, int BH, int64_t rows, int cols, int64_t r0, int64_t r1, hipStream_t s) {
  if (r1 <= r0) return LACT_OK;
  return timed(LACT_KCLASS_PREP, 0.0, s,
               [&] { return launch_zero_f32(x, BH, rows * cols, r0 * cols, (r1 - r0) * cols, s); });
}

// Rows of [0, n) that no range of `r` covers, as [b, e) pairs.
std::vector<std::pair<int64_t, int64_t>> uncovered(std::vector<std::pair<int64_t, int64_t>> r, int64_t n) {
  std::sort(r.begin(), r.end());
  std::vector<std::pair<int64_t, int64_t>> gaps;
  int64_t at = 0;
  for (const auto& x : r) {
    if (x.first > at) gaps.emplace_back(at, x.first);
    at = std::max(at, x.second);
  }
  if (n > at) gaps.emplace_back(at, n);
  return gaps;
}

// ---------------------------------------------------------------- backward
// Reverse of the linear fast weight's chunk loop (§5.4 with the §3.1 chunk
// gradient and the per-row norm-preserving update of §3.2). The linear
// gradient does not depend on the fast weight, so the negated gradients
// P_c = sum_{t in c} eta_t v_t k_t^T of all chunks come from one
// contraction (its token splits are the chunks), beside the apply's
// contributions A_c = dO_c^T Q_c; the weights W_1 .. W_nch at the chunk
// boundaries follow from one row-wise update per chunk, and their
// transposed operand copies from one launch. The reverse then walks the
// chunks from the last, carrying the cotangent of the fast weight in dW0:
// per chunk the row-wise reverse of the update, one launch of three
// products (dv before its rate, dk and dq) and a token step.
// Workspace: eta k of every key token, P and A of every chunk, the
// trajectory, the transposed copies, the partials of the tail's dO^T Q and
// the two operand copies of the update's cotangent.
struct BwdLayout {
  Plan p;
  NsBwdLayout ns;       // with Muon: the Newton-Schulz reverse's buffers
  int64_t nch;          // chunks of the forward
  bool batched;         // chunk = whole 32-token steps: one split per chunk
  int64_t group;        // chunks per launch of the batched contractions
  int64_t tail_len;     // tokens per piece of the apply-only tail
  int64_t tail_split;   // tokens per split of a tail piece (at most p.nsplit splits)
  size_t off_ek, off_P, off_A, off_traj, off_wt, off_tail, off_ub, off_ut, total;
  bool mom;             // momentum: the state's trajectory, chunk means, buffers of its reverse
  size_t off_mtraj, off_bbar_all, off_mu, off_mpart;
};

constexpr int kMomBlocks = 64;   // workgroups per instance of the momentum reverse

// nupd: the schedule's updates (negative: lact_forward's chunks); apply_len:
// its longest apply-only segment (negative: the tail n_q - n_kv).
int bwd_layout(const lact_desc* dsc, BwdLayout* L, bool mom = false, int64_t nupd = -1, int64_t apply_len = -1) {
  int rc = check_desc(dsc);
  if (rc) return rc;
  if (dsc->fast_weight != LACT_FW_LINEAR) return LACT_EUNSUPPORTED;
  L->p = make_plan(dsc);
  const Plan& p = L->p;
  const double dd = (double)p.d * p.d;
  L->nch = nupd >= 0 ? nupd : (dsc->n_kv > 0 ? cdiv(dsc->n_kv, dsc->chunk) : 0);
  // per chunk: P, A and W (fp32) and a transposed copy; per key token eta k
  const double need = (double)L->nch * p.BH * dd * (12.0 + p.esz) + (double)p.BH * dsc->n_kv * p.d * p.esz;
  if (need > 4.0e18) return LACT_EUNSUPPORTED;
  L->batched = dsc->chunk % 32 == 0;
  const TileShape g2 = bwd_tile(BWD_GRAD2, p.bf16, p.narrow);
  const int64_t tiles = (int64_t)p.BH * cdiv(p.d, g2.rows) * cdiv(p.d, g2.cols);
  L->group = std::max<int64_t>(1, ((int64_t)1 << 29) / tiles);   // two segments stay under 2^30 blocks
  L->tail_len = std::max<int64_t>(p.C, 8192);
  L->tail_split = std::max<int64_t>(32, cdiv(cdiv(L->tail_len, p.nsplit), 32) * 32);
  const size_t w4 = (size_t)p.BH * p.d * p.d * 4, wio = (size_t)p.BH * p.d * p.d * p.esz;
  size_t o = 0;
  L->off_ek = o;
  o = align_up(o + (size_t)p.BH * dsc->n_kv * p.d * p.esz);
  L->off_P = o;
  o = align_up(o + (size_t)L->nch * w4);
  L->off_A = o;
  o = align_up(o + (size_t)L->nch * w4);
  L->off_traj = o;
  o = align_up(o + (size_t)L->nch * w4);
  L->off_wt = o;
  o = align_up(o + (size_t)(L->nch + 1) * wio);
  L->off_tail = o;
  o = align_up(o + ((apply_len >= 0 ? apply_len : dsc->n_q - dsc->n_kv) > 0 ? (size_t)p.nsplit * w4 : 0));
  L->off_ub = o;
  o = align_up(o + wio);
  L->off_ut = o;
  o = align_up(o + wio);
  if (p.muon) o = ns_bwd_layout(p, dsc->ns_steps, o, &L->ns, L->nch);
  L->mom = mom;
  if (mom) {
    L->off_mtraj = o;
    o = align_up(o + (size_t)L->nch * w4);
    L->off_bbar_all = o;
    o = align_up(o + (size_t)p.BH * std::max<int64_t>(L->nch, 1) * 4);
    L->off_mu = o;
    o = align_up(o + w4);
    L->off_mpart = o;
    o = align_up(o + (size_t)p.BH * kMomBlocks * 4);
  }
  L->total = std::max<size_t>(o, kAlign);
  return LACT_OK;
}

// One GRAD2 segment: out[m][j] = sum over rows [0, n) of a[., m] b[., j], in
// splits of split_len tokens (fp32, BH d^2 floats between splits).
void lin_grad_seg(BwdSeg& g, const Plan& p, Operand a, Operand b, float* out, int64_t n, int64_t split_len) {
  const TileShape t = bwd_tile(BWD_GRAD2, p.bf16, p.narrow);
  g.kind = BWD_GRAD2;
  g.tiles_m = (int)cdiv(p.d, t.rows);
  g.tiles_n = (int)cdiv(p.d, t.cols);
  g.nsplit = (int)std::max<int64_t>(1, cdiv(n, split_len));
  g.nblocks = p.BH * g.tiles_m * g.tiles_n * g.nsplit;
  g.rows = n;
  g.split_len = split_len;
  g.a0 = a;
  g.b0 = b;
  g.out = out;
  g.out_inst = (int64_t)p.d * p.d;
  g.out_split = (int64_t)p.BH * p.d * p.d;
  g.out_off = 0;
}

// One OUT segment: out[t][m] = sum_e a[t][e] b[m][e] for rows t in [0, n)
// (rows of out d apart, instances out_inst apart).
void lin_out_seg(BwdSeg& o, const Plan& p, Operand a, Operand b, void* out, int64_t out_inst, int64_t n) {
  const TileShape t = bwd_tile(BWD_OUT, p.bf16, p.narrow);
  o.kind = BWD_OUT;
  o.tiles_m = (int)cdiv(p.d, t.rows);
  o.tiles_n = (int)cdiv(n, t.cols);
  o.nsplit = 1;
  o.nblocks = p.BH * o.tiles_m * o.tiles_n;
  o.rows = n;
  o.a0 = a;
  o.b0 = b;
  o.out = out;
  o.out_inst = out_inst;
}

int lin_launch(const Plan& p, hipStream_t s, BwdArgs& b, int nseg, double flops) {
  b.nseg = nseg;
  b.total_blocks = 0;
  for (int i = 0; i < nseg; ++i) b.total_blocks += b.seg[i].nblocks;
  b.d = p.d;
  b.h = p.d;
  b.narrow = p.narrow;
  return timed(LACT_KCLASS_BWD, flops, s, [&] { return launch_bwd(b, p.bf16, s); });
}

// With M0 != nullptr: the momentum optimizer (beta the per-token factors,
// dMf the final state's cotangent or nullptr, dbeta and dM0 the outputs).
int run_backward_linear(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                        const float* W0, const void* dout, const float* dWf, void* dq, void* dk, void* dv,
                        float* deta, float* dW0, void* workspace, size_t workspace_bytes, void* stream,
                        const float* beta = nullptr, const float* M0 = nullptr, const float* dMf = nullptr,
                        float* dbeta = nullptr, float* dM0 = nullptr, const lact_segment* sched = nullptr,
                        int64_t nsched = -1) {
  const bool mom = M0 != nullptr;
  int rc = check_desc(desc);
  if (rc) return rc;
  std::vector<BSeg> segs;
  int64_t nupd = 0, longest_apply = 0;
  rc = backward_segments(desc, sched, nsched, &segs, &nupd, &longest_apply);
  if (rc) return rc;
  BwdLayout L;
  rc = bwd_layout(desc, &L, mom, nsched >= 0 ? nupd : -1, nsched >= 0 ? longest_apply : -1);
  if (rc) return rc;
  const bool any_kv = desc->n_kv > 0, any_q = desc->n_q > 0;
  if (mom) {
    if (!dM0) return LACT_EINVAL;
    if (any_kv && (!beta || !dbeta)) return LACT_EINVAL;
    if (misaligned(M0) || misaligned(dM0) || (dMf && misaligned(dMf))) return LACT_EALIGN;
    if (any_kv && (((uintptr_t)beta & 3) || ((uintptr_t)dbeta & 3))) return LACT_EALIGN;
  }
  if (!W0 || !dW0) return LACT_EINVAL;
  if (any_q && (!q || !dout || !dq)) return LACT_EINVAL;
  if (any_kv && (!k || !v || !eta || !dk || !dv || !deta)) return LACT_EINVAL;
  if (misaligned(W0) || misaligned(dW0) || (dWf && misaligned(dWf))) return LACT_EALIGN;
  if (any_q && (misaligned(q) || misaligned(dout) || misaligned(dq))) return LACT_EALIGN;
  if (any_kv && (misaligned(k) || misaligned(v) || misaligned(dk) || misaligned(dv))) return LACT_EALIGN;
  if (any_kv && (((uintptr_t)eta & 3) || ((uintptr_t)deta & 3))) return LACT_EALIGN;
  if (!workspace || workspace_bytes < L.total) return LACT_EWORKSPACE;
  if ((uintptr_t)workspace & (kAlign - 1)) return LACT_EALIGN;
  const Plan& p = L.p;
  const hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  const int64_t n_kv = desc->n_kv, n_q = desc->n_q, C = desc->chunk, d = p.d, BH = p.BH;
  const int64_t dd = d * d, esz = p.esz, wio = BH * dd * esz;
  const size_t w4 = (size_t)BH * dd * 4;
  const int64_t psplit = BH * dd;
  const uint8_t* qb = (const uint8_t*)q;
  const uint8_t* kb = (const uint8_t*)k;
  const uint8_t* vb = (const uint8_t*)v;
  const uint8_t* ob = (const uint8_t*)dout;
  uint8_t* ek = ws + L.off_ek;
  float* Pall = reinterpret_cast<float*>(ws + L.off_P);
  float* Aall = reinterpret_cast<float*>(ws + L.off_A);
  auto traj = [&](int64_t i) -> float* {
    return i == 0 ? const_cast<float*>(W0) : reinterpret_cast<float*>(ws + L.off_traj + (size_t)(i - 1) * w4);
  };
  auto wt = [&](int64_t i) -> uint8_t* { return ws + L.off_wt + (size_t)i * wio; };
  auto mtraj = [&](int64_t i) -> float* {   // momentum state entering chunk i
    return i == 0 ? const_cast<float*>(M0) : reinterpret_cast<float*>(ws + L.off_mtraj + (size_t)(i - 1) * w4);
  };
  float* bbar_all = mom ? reinterpret_cast<float*>(ws + L.off_bbar_all) : nullptr;
  float* mu = mom ? reinterpret_cast<float*>(ws + L.off_mu) : nullptr;
  if (mom && L.nch > 0) {   // every update's mean of beta, [BH][nch]
    for (const BSeg& g : segs) {   // lact_forward's chunks: all in one launch
      if (!is_update(g.mode) || (nsched < 0 && g.before > 0)) continue;
      BetaArgs ba{};
      ba.beta = beta;
      ba.n_kv = n_kv;
      ba.chunk = nsched < 0 ? C : g.e - g.b;
      ba.t0 = nsched < 0 ? 0 : g.b;
      ba.end = nsched < 0 ? n_kv : g.e;
      ba.nchunks = nsched < 0 ? (int)L.nch : 1;
      ba.BH = p.BH;
      ba.bbar = bbar_all + (nsched < 0 ? 0 : g.before);
      ba.stride = (int)L.nch;
      rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_beta_mean(ba, s); });
      if (rc) return rc;
    }
  }
  if (nsched >= 0) {   // rows of the cotangents that no apply or no update reaches
    std::vector<std::pair<int64_t, int64_t>> ur, ar;
    for (const BSeg& g : segs) {
      if (is_update(g.mode)) ur.emplace_back(g.b, g.e);
      if (is_apply(g.mode)) ar.emplace_back(g.b, g.e);
    }
    for (const auto& gap : uncovered(ar, n_q)) {
      rc = timed(LACT_KCLASS_PREP, 0.0, s,
                 [&] { return launch_zero_rows(dq, p.BH, d * esz, n_q, gap.first, gap.second, s); });
      if (rc) return rc;
    }
    for (const auto& gap : uncovered(ur, n_kv)) {
      rc = timed(LACT_KCLASS_PREP, 0.0, s,
                 [&] { return launch_zero_rows(dk, p.BH, d * esz, n_kv, gap.first, gap.second, s); });
      if (!rc) rc = timed(LACT_KCLASS_PREP, 0.0, s,
                          [&] { return launch_zero_rows(dv, p.BH, d * esz, n_kv, gap.first, gap.second, s); });
      if (!rc) rc = zero_f32_rows(deta, p.BH, n_kv, 1, gap.first, gap.second, s);
      if (!rc && mom) rc = zero_f32_rows(dbeta, p.BH, n_kv, 1, gap.first, gap.second, s);
      if (rc) return rc;
    }
  }
  // eta k of every key token, then P_c and A_c of every chunk (of every
  // update segment, and the apply of the same tokens when it has one)
  if (any_kv) {
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
      return launch_scale_rows(kb, eta, ek, p.BH, n_kv, p.d, n_kv * d, n_kv, n_kv * d, p.bf16, s);
    });
    if (rc) return rc;
  }
  if (nsched >= 0) {
    for (const BSeg& g : segs) {
      if (!is_update(g.mode)) continue;
      const int64_t t0 = g.b, n = g.e - g.b, one = cdiv(n, 32) * 32, u = g.before;
      BwdArgs b{};
      lin_grad_seg(b.seg[0], p, op(vb + t0 * d * esz, d, n_kv * d), op(ek + t0 * d * esz, d, n_kv * d),
                   Pall + u * psplit, n, one);
      const bool app = is_apply(g.mode);
      if (app)
        lin_grad_seg(b.seg[1], p, op(ob + t0 * d * esz, d, n_q * d), op(qb + t0 * d * esz, d, n_q * d),
                     Aall + u * psplit, n, one);
      rc = lin_launch(p, s, b, app ? 2 : 1, (app ? 4.0 : 2.0) * BH * n * dd);
      if (rc) return rc;
    }
  } else if (L.batched) {
    for (int64_t c0 = 0; c0 < L.nch; c0 += L.group) {
      const int64_t t0 = c0 * C, t1 = std::min(n_kv, (c0 + L.group) * C), n = t1 - t0;
      BwdArgs b{};
      lin_grad_seg(b.seg[0], p, op(vb + t0 * d * esz, d, n_kv * d), op(ek + t0 * d * esz, d, n_kv * d),
                   Pall + c0 * psplit, n, C);
      lin_grad_seg(b.seg[1], p, op(ob + t0 * d * esz, d, n_q * d), op(qb + t0 * d * esz, d, n_q * d),
                   Aall + c0 * psplit, n, C);
      rc = lin_launch(p, s, b, 2, 4.0 * BH * n * dd);
      if (rc) return rc;
    }
  } else {
    for (int64_t ci = 0; ci < L.nch; ++ci) {
      const int64_t t0 = ci * C, n = std::min(n_kv, t0 + C) - t0, one = cdiv(n, 32) * 32;
      BwdArgs b{};
      lin_grad_seg(b.seg[0], p, op(vb + t0 * d * esz, d, n_kv * d), op(ek + t0 * d * esz, d, n_kv * d),
                   Pall + ci * psplit, n, one);
      lin_grad_seg(b.seg[1], p, op(ob + t0 * d * esz, d, n_q * d), op(qb + t0 * d * esz, d, n_q * d),
                   Aall + ci * psplit, n, one);
      rc = lin_launch(p, s, b, 2, 4.0 * BH * n * dd);
      if (rc) return rc;
    }
  }
  // W_{c+1} = rows of W_c + P_c (or, with Muon, W_c - Muon(g_c)) rescaled to
  // W_c's row norms; with momentum the step is M_{c+1} = bbar_c M_c + g_c
  // (or Muon of it)
  for (int64_t ci = 0; ci < L.nch; ++ci) {
    UpdArgs u{};
    u.W[0] = traj(ci + 1);
    u.Wsrc[0] = traj(ci);
    u.step = Pall + ci * psplit;
    if (mom && !p.muon) {   // the update advances the state in place, in its trajectory slot
      rc = timed(LACT_KCLASS_PREP, 0.0, s,
                 [&] { return hipMemcpyAsync(mtraj(ci + 1), mtraj(ci), w4, hipMemcpyDeviceToDevice, s); });
      if (rc) return rc;
      u.M[0] = mtraj(ci + 1);
      u.bbar = bbar_all + ci;
      u.bbar_stride = (int)L.nch;
    }
    if (p.muon) {   // the iterates go to this chunk's slice when they are kept
      const NsBwd nb{p, L.ns, ws, s, desc->ns_steps, {p.d, 0, 0}, {p.d, 0, 0}, ci};
      const float* slab[3] = {mtraj(ci + 1), nullptr, nullptr};
      if (mom) {
        rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
          return launch_mom_adv(mtraj(ci), bbar_all + ci, L.nch, PartSet{Pall + ci * psplit, 1, psplit, dd},
                                mtraj(ci + 1), p.BH, dd, s);
        });
        if (rc) return rc;
      }
      rc = nb.forward(Pall + ci * psplit, 1, psplit, mom ? slab : nullptr);
      if (rc) return rc;
      u.step = nb.pst();
    }
    u.nsplit = 1;
    u.step_split = 0;
    u.nmat = 1;
    u.BH = p.BH;
    u.d = p.d;
    u.h = p.d;
    u.rows_total = p.BH * p.d;
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_update(u, false, s); });
    if (rc) return rc;
  }
  // transposed operand copies of W_0 .. W_nch (W_1 .. W_nch are contiguous)
  {
    const CopySeg cs{W0, dd, p.d, p.d, nullptr, 0, 0, wt(0), d, dd};
    rc = timed(LACT_KCLASS_PREP, 0.0, s, [&] { return launch_copies(&cs, 1, p.BH, p.bf16, s); });
  }
  if (rc) return rc;
  {
    const int64_t t = cdiv(d, 32), per = std::max<int64_t>(1, ((int64_t)1 << 30) / (BH * t * t));
    for (int64_t c0 = 1; c0 <= L.nch; c0 += per) {   // whole sets of BH matrices, under 2^30 blocks
      const int64_t m = std::min(per, L.nch + 1 - c0);
      const CopySeg cs{traj(c0), dd, p.d, p.d, nullptr, 0, 0, wt(c0), d, dd};
      rc = timed(LACT_KCLASS_PREP, 0.0, s, [&] { return launch_copies(&cs, 1, (int)(m * BH), p.bf16, s); });
      if (rc) return rc;
    }
  }
  float* G = dW0;
  // The cotangent of the current weight lives in G; `first` while it still
  // has to start from dW_final (or zero).
  bool first = true;
  auto add_g = [&](PartSet ps) -> int {
    const int mode = first ? (dWf ? 1 : 0) : 2;
    first = false;
    return timed(LACT_KCLASS_UPDATE, 0.0, s,
                 [&] { return launch_accum(G, dd, dWf, dd, mode, ps, PartSet{}, p.BH, dd, s); });
  };
  if (mom) {   // the final state's cotangent, or zero
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s,
               [&] { return launch_accum(dM0, dd, dMf, dd, dMf ? 1 : 0, PartSet{}, PartSet{}, p.BH, dd, s); });
    if (rc) return rc;
  }
  uint8_t* ub = ws + L.off_ub;
  uint8_t* ut = ws + L.off_ut;
  for (auto it = segs.rbegin(); it != segs.rend(); ++it) {
    const BSeg& g = *it;
    if (g.mode == LACT_SEG_APPLY_ONLY) {   // applied with the weight of its time, in pieces
      float* tpart = reinterpret_cast<float*>(ws + L.off_tail);
      for (int64_t a = g.b; a < g.e; a += L.tail_len) {
        const int64_t n = std::min(L.tail_len, g.e - a);
        BwdArgs b{};
        lin_grad_seg(b.seg[0], p, op(ob + a * d * esz, d, n_q * d), op(qb + a * d * esz, d, n_q * d), tpart, n,
                     L.tail_split);
        lin_out_seg(b.seg[1], p, op(ob + a * d * esz, d, n_q * d), op(wt(g.before), d, dd),
                    (uint8_t*)dq + a * d * esz, n_q * d, n);
        rc = lin_launch(p, s, b, 2, 4.0 * BH * n * dd);
        if (!rc) rc = add_g(PartSet{tpart, b.seg[0].nsplit, psplit, dd});
        if (rc) return rc;
      }
      continue;
    }
    if (first) {
      rc = add_g(PartSet{});
      if (rc) return rc;
    }
    const int64_t ci = g.before, s0 = g.b, n = g.e - g.b;
    const bool then_apply = g.mode == LACT_SEG_UPDATE_THEN_APPLY;
    const bool applies = g.mode != LACT_SEG_UPDATE_ONLY;
    const NsBwd nb{p, L.ns, ws, s, desc->ns_steps, {p.d, 0, 0}, {p.d, 0, 0}, ci};
    const float* slab[3] = {mom ? mtraj(ci + 1) : nullptr, nullptr, nullptr};
    if (p.muon) {   // the step is Muon(g), or Muon(M_{c+1}): its kept iterates, else replay the iteration
      rc = nb.kept() ? nb.prepare(Pall + ci * psplit, 1, psplit, mom ? slab : nullptr)
                     : nb.forward(Pall + ci * psplit, 1, psplit, mom ? slab : nullptr);
      if (rc) return rc;
    }
    VjpArgs va{};
    va.W = traj(ci);
    va.w_inst = dd;
    va.P = p.muon ? PartSet{nb.pst(), 1, psplit, dd}
                  : (mom ? PartSet{mtraj(ci + 1), 1, 0, dd, -1.0f} : PartSet{Pall + ci * psplit, 1, psplit, dd});
    const PartSet ac{Aall + ci * psplit, 1, psplit, dd};
    if (applies && then_apply) va.pre[0] = ac;   // applied with the weights leaving the update
    else if (applies) va.post = ac;
    va.G = G;
    va.g_inst = dd;
    va.Ub = ub;
    va.ub_ld = d;
    va.ub_inst = dd;
    va.UT = ut;
    va.ut_ld = d;
    va.ut_inst = dd;
    va.BH = p.BH;
    va.R = p.d;
    va.L = p.d;
    if (p.muon || mom) {   // the update's cotangent in fp32 (Newton-Schulz or momentum reverse next)
      va.Ub = va.UT = nullptr;
      va.U32 = p.muon ? nb.at<float>(L.ns.ustep) : mu;
      va.u32_inst = dd;
    }
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_vjp(&va, 1, p.bf16, s); });
    if (rc) return rc;
    if (p.muon) {
      rc = nb.reverse();
      if (rc) return rc;
    }
    const float* ug = p.muon ? nb.at<float>(L.ns.ug) : mu;
    if (mom) {   // dM' = carried - (step's share); the gradient's cotangent; carry bbar dM'; dbeta
      MomBwdArgs ma{};
      ma.U = const_cast<float*>(ug);
      ma.R[0] = dM0;
      ma.M[0] = mtraj(ci);
      ma.bbar = bbar_all + ci;
      ma.bbar_inst = L.nch;
      ma.part = reinterpret_cast<float*>(ws + L.off_mpart);
      ma.BH = p.BH;
      ma.nmat = 1;
      ma.nblk = kMomBlocks;
      ma.dh = dd;
      rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_mom_bwd(ma, s); });
      if (!rc) rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
        return launch_mom_dbeta(ma.part, kMomBlocks, p.BH, dbeta + s0, n_kv, n, s);
      });
      if (rc) return rc;
    }
    if (p.muon || mom) {   // the gradient's cotangent (negated) in the operand layouts
      const CopySeg cs{ug, dd, p.d, p.d, ub, d, dd, ut, d, dd};
      rc = timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_copies(&cs, 1, p.BH, p.bf16, s); });
      if (rc) return rc;
    }
    BwdArgs b{};
    lin_out_seg(b.seg[0], p, op(kb + s0 * d * esz, d, n_kv * d), op(ub, d, dd), (uint8_t*)dv + s0 * d * esz,
                n_kv * d, n);   // Y = K Uh^T
    lin_out_seg(b.seg[1], p, op(vb + s0 * d * esz, d, n_kv * d), op(ut, d, dd), (uint8_t*)dk + s0 * d * esz,
                n_kv * d, n);   // dk = eta (V Uh)
    b.seg[1].row_scale = eta + s0;
    b.seg[1].scale_inst = n_kv;
    // dq = dO W with the weight the chunk was applied with
    lin_out_seg(b.seg[2], p, op(ob + s0 * d * esz, d, n_q * d), op(wt(then_apply ? ci + 1 : ci), d, dd),
                (uint8_t*)dq + s0 * d * esz, n_q * d, n);
    rc = lin_launch(p, s, b, applies ? 3 : 2, (applies ? 6.0 : 4.0) * BH * n * dd);
    if (rc) return rc;
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
      return launch_lin_tokens(vb + s0 * d * esz, eta + s0, (uint8_t*)dv + s0 * d * esz, deta + s0, p.BH, n, p.d,
                               n_kv * d, n_kv, p.bf16, s);
    });
    if (rc) return rc;
  }
  if (first) return add_g(PartSet{});   // no update: dW_final (or zero)
  return LACT_OK;
}

// Reverse of the SwiGLU fast weight's chunk loop (§3.1 loss and chunk
// gradient, §3.2 per-row norm-preserving update; Alg. 1), one rate per token
// or one per matrix (Alg. 1's three rates), with Muon (NsBwd) and the
// momentum optimizer (App. A) optional. The forward's own update launches replay
// the chunk loop (unfused, so that every chunk's negated gradient P_c stays
// in a slot of its own, and reading W_c from the trajectory while writing
// W_{c+1}). The reverse then walks the chunks from the last, carrying the
// cotangent of (W1, W2, W3) in dW1, dW2, dW3. Per chunk: the row-wise reverse
// of the update (three matrices, one launch), the operand copies of the
// chunk's weights (one launch), nine [n x h] products in three launches
// (Z1 = K W1^T, Z3 = K W3^T, C = V W2; the same with the update's cotangent;
// the apply's Q W1^T, Q W3^T, dO W2), the per-token steps with SiLU's first
// and second derivatives, one launch for dk (a sum over 4h), dv and dq (over
// 2h), and the weight cotangents of the gradient's own dependence on W and
// of the apply (GRAD13 + GRAD2, two launches). The contractions are the OUT
// and GRAD kinds with operands laid out so that each sum runs over one
// contiguous row ([R3 | R1 | dZ1 | dZ3] against [U3^T | U1^T | W1^T | W3^T],
// [eta A | dC] against [U2 | W2], [dZq1 | dZq3] against [W1^T | W3^T]).
struct SwBwdLayout {
  Plan p;               // the forward's plan without the fused gradient-and-update kind
  NsBwdLayout ns;       // with Muon: the Newton-Schulz reverse's buffers
  bool mom;             // momentum: the state's trajectory, chunk means, buffers of its reverse
  size_t off_mtraj, off_bbar_all, off_mu, off_mpart;
  int64_t nch;          // updates of the forward (its chunks, or the schedule's update segments)
  int64_t T;            // token rows of the chunk buffers (a chunk, or a piece of an apply-only stretch)
  int64_t tail_split;   // tokens per split of a tail piece (at most p.nsplit splits)
  size_t slotP;         // bytes of one chunk's gradient partials
  size_t off_P, off_traj, off_z[6], off_pk, off_pv, off_pq, off_hq, off_u[3], off_a[3], off_bk, off_bv, off_bq,
      off_ur[3], off_apart, off_bpart, total;
  size_t off_keep, keep_slot;   // per update: the replay's Z1, Z3, D ([BH][chunk][h] each, io dtype)
};

// nupd: the schedule's updates (negative: lact_forward's chunks);
// apply_len: its longest apply-only segment (negative: the tail n_q - n_kv).
int sw_bwd_layout(const lact_desc* dsc, SwBwdLayout* L, bool mom = false, int64_t nupd = -1,
                  int64_t apply_len = -1) {
  int rc = check_desc(dsc);
  if (rc) return rc;
  if (dsc->fast_weight != LACT_FW_SWIGLU) return LACT_EUNSUPPORTED;
  L->p = make_plan(dsc, false);
  const Plan& p = L->p;
  const double dh = (double)p.d * p.h;
  L->nch = nupd >= 0 ? nupd : (dsc->n_kv > 0 ? cdiv(dsc->n_kv, dsc->chunk) : 0);
  const int64_t tail = apply_len >= 0 ? apply_len : dsc->n_q - dsc->n_kv;
  L->T = std::max<int64_t>(1, std::max<int64_t>(p.C, std::min<int64_t>(tail, 4096)));
  const double need = (double)L->nch * p.BH * dh * 12.0 * (p.nsplit + 1) + (double)p.BH * L->T * p.h * p.esz * 15.0 +
                      (double)L->nch * 3 * p.BH * p.C * p.h * p.esz;
  if (need > 4.0e18) return LACT_EUNSUPPORTED;
  L->tail_split = std::max<int64_t>(32, cdiv(cdiv(L->T, p.nsplit), 32) * 32);
  const size_t w4 = (size_t)p.BH * p.d * p.h * 4, wio = (size_t)p.BH * p.d * p.h * p.esz;
  const size_t rows = (size_t)p.BH * L->T * p.h * p.esz;   // one [T x h] buffer
  L->slotP = (size_t)p.nsplit * 3 * w4;
  // the forward's own layout first (at least what its validation asks for)
  size_t o = align_up(std::max(p.total, make_plan(dsc).total));
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L->off_P = take((size_t)L->nch * L->slotP);
  L->off_traj = take((size_t)L->nch * 3 * w4);
  for (int i = 0; i < 6; ++i) L->off_z[i] = take(rows);
  L->off_pk = take(4 * rows);   // [T x 4h]: R3 | R1 | dZ1 | dZ3
  L->off_pv = take(2 * rows);   // [T x 2h]: eta A | dC
  L->off_pq = take(2 * rows);   // [T x 2h]: dZq1 | dZq3
  L->off_hq = take(rows);       // [T x h]: the apply's hidden
  for (int i = 0; i < 3; ++i) L->off_u[i] = take(wio);   // W1, W3 row-major and W2^T of the update's weights
  for (int i = 0; i < 3; ++i) L->off_a[i] = take(wio);   // the same of the apply's weights
  L->off_bk = take(4 * wio);    // [d x 4h]: U3^T | U1^T | W1^T | W3^T
  L->off_bv = take(2 * wio);    // [d x 2h]: U2 | W2
  L->off_bq = take(2 * wio);    // [d x 2h]: W1^T | W3^T of the apply's weights
  for (int i = 0; i < 3; ++i) L->off_ur[i] = take(wio);   // U1, U3 row-major and U2^T
  L->off_apart = take((size_t)p.nsplit * 3 * w4);
  L->off_bpart = take((size_t)p.nsplit * 3 * w4);
  L->keep_slot = align_up((size_t)3 * p.BH * p.C * p.h * p.esz);
  L->off_keep = take((size_t)L->nch * L->keep_slot);
  if (p.muon) o = ns_bwd_layout(p, dsc->ns_steps, o, &L->ns, L->nch);
  L->mom = mom;
  if (mom) {
    L->off_mtraj = take((size_t)L->nch * 3 * w4);
    L->off_bbar_all = take((size_t)p.BH * std::max<int64_t>(L->nch, 1) * 4);
    L->off_mu = take(3 * w4);
    L->off_mpart = take((size_t)p.BH * kMomBlocks * 4);
  }
  L->total = o;
  return LACT_OK;
}

// With beta != nullptr: the momentum optimizer (M0 the initial state, dMf
// the final state's cotangents or nullptr, dbeta and dM the outputs). With
// nsched >= 0: the caller's schedule `sched` (else lact_forward's chunks).
int run_backward_swiglu(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                        const float* const W0[3], const void* dout, const float* const dWf[3], void* dq, void* dk,
                        void* dv, float* deta, float* const dW[3], void* workspace, size_t workspace_bytes,
                        void* stream, const float* beta = nullptr, const float* const* M0 = nullptr,
                        const float* const* dMf = nullptr, float* dbeta = nullptr, float* const* dMo = nullptr,
                        const lact_segment* sched = nullptr, int64_t nsched = -1) {
  const bool mom = M0 != nullptr;
  int rc = check_desc(desc);
  if (rc) return rc;
  std::vector<BSeg> segs;
  int64_t nupd = 0, longest_apply = 0;
  rc = backward_segments(desc, sched, nsched, &segs, &nupd, &longest_apply);
  if (rc) return rc;
  SwBwdLayout L;
  rc = sw_bwd_layout(desc, &L, mom, nupd, longest_apply);
  if (rc) return rc;
  const bool any_kv = desc->n_kv > 0, any_q = desc->n_q > 0;
  if (mom) {
    for (int m = 0; m < 3; ++m) {
      if (!M0[m] || !dMo[m]) return LACT_EINVAL;
      if (misaligned(M0[m]) || misaligned(dMo[m]) || (dMf[m] && misaligned(dMf[m]))) return LACT_EALIGN;
    }
    if (any_kv && (!beta || !dbeta)) return LACT_EINVAL;
    if (any_kv && (((uintptr_t)beta & 3) || ((uintptr_t)dbeta & 3))) return LACT_EALIGN;
  }
  for (int m = 0; m < 3; ++m) {
    if (!W0[m] || !dW[m]) return LACT_EINVAL;
    if (misaligned(W0[m]) || misaligned(dW[m]) || (dWf[m] && misaligned(dWf[m]))) return LACT_EALIGN;
  }
  if (any_q && (!q || !dout || !dq)) return LACT_EINVAL;
  if (any_kv && (!k || !v || !eta || !dk || !dv || !deta)) return LACT_EINVAL;
  if (any_q && (misaligned(q) || misaligned(dout) || misaligned(dq))) return LACT_EALIGN;
  if (any_kv && (misaligned(k) || misaligned(v) || misaligned(dk) || misaligned(dv))) return LACT_EALIGN;
  if (any_kv && (((uintptr_t)eta & 3) || ((uintptr_t)deta & 3))) return LACT_EALIGN;
  if (!workspace || workspace_bytes < L.total) return LACT_EWORKSPACE;
  if ((uintptr_t)workspace & (kAlign - 1)) return LACT_EALIGN;
  Ctx c;
  // the forward's context; its updates read W_u and write W_{u+1} in the
  // trajectory, never W0
  float* const Mseed[3] = {mom ? const_cast<float*>(M0[0]) : nullptr, mom ? const_cast<float*>(M0[1]) : nullptr,
                           mom ? const_cast<float*>(M0[2]) : nullptr};
  rc = setup(c, desc, q, k, v, eta, mom ? beta : nullptr, const_cast<float*>(W0[0]), const_cast<float*>(W0[1]),
             const_cast<float*>(W0[2]), mom ? Mseed : nullptr, dq, workspace, workspace_bytes, stream);
  if (rc) return rc;
  c.p = L.p;
  const Plan& p = c.p;
  const hipStream_t s = c.s;
  uint8_t* ws = c.ws;
  const int64_t n_kv = desc->n_kv, n_q = desc->n_q, d = p.d, h = p.h, BH = p.BH;
  const int64_t dh = d * h, esz = p.esz;
  const size_t w4 = (size_t)BH * dh * 4;
  const int64_t psplit = BH * 3 * dh;   // floats between splits of a partial set
  auto traj = [&](int64_t i, int m) -> float* {   // weights entering update i (i = nupd: the final ones)
    return i == 0 ? const_cast<float*>(W0[m])
                  : reinterpret_cast<float*>(ws + L.off_traj + ((size_t)(i - 1) * 3 + m) * w4);
  };
  auto mtraj = [&](int64_t i, int m) -> float* {   // momentum state entering update i
    return i == 0 ? const_cast<float*>(M0[m])
                  : reinterpret_cast<float*>(ws + L.off_mtraj + ((size_t)(i - 1) * 3 + m) * w4);
  };
  // rows of the cotangents that no apply (dq) or no update (dk, dv, deta, dbeta) reaches
  if (nsched >= 0) {
    std::vector<std::pair<int64_t, int64_t>> ur, ar;
    for (const BSeg& g : segs) {
      if (is_update(g.mode)) ur.emplace_back(g.b, g.e);
      if (is_apply(g.mode)) ar.emplace_back(g.b, g.e);
    }
    for (const auto& gap : uncovered(ar, n_q)) {
      rc = timed(LACT_KCLASS_PREP, 0.0, s,
                 [&] { return launch_zero_rows(dq, p.BH, d * esz, n_q, gap.first, gap.second, s); });
      if (rc) return rc;
    }
    for (const auto& gap : uncovered(ur, n_kv)) {
      rc = timed(LACT_KCLASS_PREP, 0.0, s,
                 [&] { return launch_zero_rows(dk, p.BH, d * esz, n_kv, gap.first, gap.second, s); });
      if (!rc) rc = timed(LACT_KCLASS_PREP, 0.0, s,
                          [&] { return launch_zero_rows(dv, p.BH, d * esz, n_kv, gap.first, gap.second, s); });
      if (!rc) rc = zero_f32_rows(deta, p.BH, n_kv, p.es, gap.first, gap.second, s);
      if (!rc && mom) rc = zero_f32_rows(dbeta, p.BH, n_kv, 1, gap.first, gap.second, s);
      if (rc) return rc;
    }
  }
  // replay: every update's weights (and state) in the trajectory, its
  // negated gradient partials in a slot of its own
  rc = prepare_weights(c);
  if (rc) return rc;
  float* bbar_all = mom ? reinterpret_cast<float*>(ws + L.off_bbar_all) : nullptr;
  for (const BSeg& g : segs) {
    if (!is_update(g.mode)) continue;
    const int64_t u = g.before;
    if (mom) {   // the update's mean of beta (the replay's slot and [BH][nupd]); the state advances in its slot
      c.chunk_idx = 0;
      rc = beta_means(c, g.b, g.e - g.b, g.e, 1);
      if (rc) return rc;
      BetaArgs ba{};
      ba.beta = beta;
      ba.n_kv = n_kv;
      ba.chunk = g.e - g.b;
      ba.t0 = g.b;
      ba.end = g.e;
      ba.nchunks = 1;
      ba.BH = p.BH;
      ba.bbar = bbar_all + u;
      ba.stride = (int)nupd;
      rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_beta_mean(ba, s); });
      if (rc) return rc;
      for (int m = 0; m < 3; ++m) {
        rc = timed(LACT_KCLASS_PREP, 0.0, c.s,
                   [&] { return hipMemcpyAsync(mtraj(u + 1, m), mtraj(u, m), w4, hipMemcpyDeviceToDevice, c.s); });
        if (rc) return rc;
        c.M[m] = mtraj(u + 1, m);
      }
    }
    const bool keep = p.muon && L.ns.iters > 1;   // the iteration runs here, once, its iterates kept
    for (int m = 0; m < 3; ++m) {
      c.W[m] = traj(u + 1, m);
      c.Wsrc[m] = traj(u, m);
      if (p.muon && !keep) {   // Muon's fused last steps update W in place: start from a copy
        c.Wsrc[m] = nullptr;
        rc = timed(LACT_KCLASS_PREP, 0.0, c.s,
                   [&] { return hipMemcpyAsync(traj(u + 1, m), traj(u, m), w4, hipMemcpyDeviceToDevice, c.s); });
        if (rc) return rc;
      }
    }
    if (!p.bf16) {   // fp32: the contractions read the state itself
      c.wop[0] = op(traj(u, 0), d, dh);
      c.wop[1] = op(traj(u, 1), h, dh);
      c.wop[2] = op(traj(u, 2), d, dh);
    }
    c.p.off_step = L.off_P + (size_t)u * L.slotP;
    c.grad_only = keep;
    for (int m = 0; m < 3; ++m) c.keep[m] = ws + L.off_keep + (size_t)u * L.keep_slot + (size_t)m * p.BH * p.C * h * esz;
    c.keep_inst = p.C * h;   // the reverse reads this update's Z1, Z3 and D from here
    rc = update_chunk(c, g.b, g.e, false);
    c.grad_only = false;
    for (int m = 0; m < 3; ++m) c.keep[m] = nullptr;
    if (rc) return rc;
    if (keep) {
      float* gslot = reinterpret_cast<float*>(ws + c.p.off_step);
      const float* mnext[3] = {mom ? mtraj(u + 1, 0) : nullptr, mom ? mtraj(u + 1, 1) : nullptr,
                               mom ? mtraj(u + 1, 2) : nullptr};
      if (mom) {   // M_{u+1} = bbar M_u + g (the copy above is overwritten)
        for (int m = 0; m < 3; ++m) {
          rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
            return launch_mom_adv(mtraj(u, m), bbar_all + u, nupd,
                                  PartSet{gslot + m * dh, p.nsplit, psplit, 3 * dh}, mtraj(u + 1, m), p.BH, dh, s);
          });
          if (rc) return rc;
        }
      }
      const NsBwd nb{p, L.ns, ws, s, desc->ns_steps, {(int)h, (int)d, (int)h}, {(int)d, (int)h, (int)d}, u};
      rc = nb.forward(gslot, p.nsplit, psplit, mom ? mnext : nullptr);
      if (rc) return rc;
      UpdArgs ua{};
      for (int m = 0; m < 3; ++m) {
        ua.W[m] = traj(u + 1, m);
        ua.Wsrc[m] = traj(u, m);
        ua.Wb[m] = p.bf16 ? c.wb[c.wset][m] : nullptr;   // fp32: the next contractions read the state
      }
      ua.step = nb.pst();
      ua.nsplit = 1;
      ua.step_split = 0;
      ua.BH = p.BH;
      ua.d = p.d;
      ua.h = p.h;
      ua.nmat = 3;
      ua.rows_total = p.BH * (2 * p.h + p.d);
      rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_update(ua, p.bf16, s); });
      if (rc) return rc;
    }
  }
  c.p.off_step = L.p.off_step;
  if (mom) {   // the final state's cotangent, or zero
    for (int m = 0; m < 3; ++m) {
      rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
        return launch_accum(dMo[m], dh, dMf[m], dh, dMf[m] ? 1 : 0, PartSet{}, PartSet{}, p.BH, dh, s);
      });
      if (rc) return rc;
    }
  }
  const uint8_t* qb = (const uint8_t*)q;
  const uint8_t* kb = (const uint8_t*)k;
  const uint8_t* vb = (const uint8_t*)v;
  const uint8_t* ob = (const uint8_t*)dout;
  uint8_t* zb[6];
  for (int i = 0; i < 6; ++i) zb[i] = ws + L.off_z[i];
  uint8_t* pk = ws + L.off_pk;
  uint8_t* pv = ws + L.off_pv;
  uint8_t* pq = ws + L.off_pq;
  uint8_t* hq = ws + L.off_hq;
  uint8_t* bk = ws + L.off_bk;
  uint8_t* bv = ws + L.off_bv;
  uint8_t* bq = ws + L.off_bq;
  uint8_t* ur[3] = {ws + L.off_ur[0], ws + L.off_ur[1], ws + L.off_ur[2]};
  float* apart = reinterpret_cast<float*>(ws + L.off_apart);
  float* bpart = reinterpret_cast<float*>(ws + L.off_bpart);
  const int64_t T = L.T;
  const int64_t zi = T * h;   // elements between instances of a [T x h] buffer
  // one launch of up to three OUT segments, out[t][m] = sum_e a[t][e] b[m][e]
  // over K columns (per segment), rows of out `rows_out` wide; `pre` holds
  // gradient segments (grads into a BwdArgs) that run first in the same launch
  struct Out {
    Operand a, b;
    void* out;
    int64_t out_inst;
    int64_t K;
  };
  struct Pending {
    BwdArgs b{};
    double fl = 0.0;
  };
  auto outs = [&](const Out* o, int nseg, int64_t n, int rows_out, const Pending* pre = nullptr) -> int {
    BwdArgs b{};
    const TileShape t = bwd_tile(BWD_OUT, p.bf16, p.narrow);
    double fl = 0.0;
    const int np = pre ? pre->b.nseg : 0;
    for (int i = 0; i < np; ++i) b.seg[i] = pre->b.seg[i];
    if (pre) fl = pre->fl;
    for (int i = 0; i < nseg; ++i) {
      BwdSeg& g = b.seg[np + i];
      g.kind = BWD_OUT;
      g.tiles_m = (int)cdiv(rows_out, t.rows);
      g.tiles_n = (int)cdiv(n, t.cols);
      g.nsplit = 1;
      g.nblocks = p.BH * g.tiles_m * g.tiles_n;
      g.rows = n;
      g.a0 = o[i].a;
      g.b0 = o[i].b;
      g.out = o[i].out;
      g.out_inst = o[i].out_inst;
      g.klen = o[i].K;
      fl += 2.0 * BH * n * rows_out * o[i].K;
    }
    b.nseg = np + nseg;
    b.total_blocks = 0;
    for (int i = 0; i < b.nseg; ++i) b.total_blocks += b.seg[i].nblocks;
    // the gradient kinds read d and h as the weights' shape; every OUT
    // segment carries its own contraction length
    b.d = np ? (int)d : rows_out;
    b.h = np ? (int)h : (int)o[0].K;
    b.narrow = p.narrow;
    return timed(LACT_KCLASS_BWD, fl, s, [&] { return launch_bwd(b, p.bf16, s); });
  };
  // weight cotangents over rows [0, n): W1 += a1^T b, W3 += a3^T b (GRAD13)
  // and W2 += a2^T b2 (GRAD2), as split partials into `out`
  auto grads = [&](Operand a1, Operand a3, Operand b13, Operand a2, Operand b2, float* out, int64_t n,
                   int64_t split_len, int* nsplit, Pending* into = nullptr) -> int {
    const TileShape g13 = bwd_tile(BWD_GRAD13, p.bf16, p.narrow), g2 = bwd_tile(BWD_GRAD2, p.bf16, p.narrow);
    const int ns = (int)std::max<int64_t>(1, cdiv(n, split_len));
    BwdArgs b{};
    BwdSeg& x = b.seg[0];
    x.kind = BWD_GRAD13;
    x.tiles_m = (int)cdiv(h, g13.rows);
    x.tiles_n = (int)cdiv(d, g13.cols);
    x.nsplit = ns;
    x.nblocks = p.BH * x.tiles_m * x.tiles_n * ns;
    x.rows = n;
    x.split_len = split_len;
    x.a0 = a1;
    x.a1 = a3;
    x.b0 = b13;
    x.out = out;
    x.out_inst = 3 * dh;
    x.out_split = psplit;
    BwdSeg& y = b.seg[1];
    y.kind = BWD_GRAD2;
    y.tiles_m = (int)cdiv(d, g2.rows);
    y.tiles_n = (int)cdiv(h, g2.cols);
    y.nsplit = ns;
    y.nblocks = p.BH * y.tiles_m * y.tiles_n * ns;
    y.rows = n;
    y.split_len = split_len;
    y.a0 = a2;
    y.b0 = b2;
    y.out = out;
    y.out_inst = 3 * dh;
    y.out_split = psplit;
    y.out_off = dh;
    b.nseg = 2;
    b.total_blocks = x.nblocks + y.nblocks;
    b.d = p.d;
    b.h = p.h;
    b.narrow = p.narrow;
    *nsplit = ns;
    if (into) {   // joins a later launch (the caller keeps the order of reads and writes)
      into->b.seg[into->b.nseg++] = x;
      into->b.seg[into->b.nseg++] = y;
      into->fl += 6.0 * BH * n * dh;
      return LACT_OK;
    }
    return timed(LACT_KCLASS_BWD, 6.0 * BH * n * dh, s, [&] { return launch_bwd(b, p.bf16, s); });
  };
  // operand copies of weights (W1, W2, W3): W1, W3 row-major and W2^T into
  // `u`, W1^T | W3^T into `bt` (ld bt_ld), and W2 into `b2` (ld 2h) if given
  auto weight_copies = [&](int64_t i, const size_t* u, uint8_t* bt, int64_t bt_ld, uint8_t* b2) -> int {
    const float* W1 = traj(i, 0);
    const float* W2 = traj(i, 1);
    const float* W3 = traj(i, 2);
    // each matrix read once, both of its copies written from the same tile
    const CopySeg cs[3] = {{W1, dh, (int)h, (int)d, ws + u[0], d, dh, bt, bt_ld, d * bt_ld},
                           {W3, dh, (int)h, (int)d, ws + u[1], d, dh, bt + h * esz, bt_ld, d * bt_ld},
                           {W2, dh, (int)d, (int)h, b2, 2 * h, d * 2 * h, ws + u[2], d, dh}};
    return timed(LACT_KCLASS_PREP, 0.0, s, [&] { return launch_copies(cs, 3, p.BH, p.bf16, s); });
  };
  int a_ns = 0, b_ns = 0;
  // the apply's reverse on query rows [a, a + n) up to its weight cotangents
  // (into apart) with the weights whose copies are in `u`; dq is left to
  // the caller's OUT launch (Pq against the transposed weights)
  auto apply_back = [&](int64_t a, int64_t n, const size_t* u, int64_t split_len, Pending* into = nullptr) -> int {
    const Operand qo = op(qb + a * d * esz, d, n_q * d), doo = op(ob + a * d * esz, d, n_q * d);
    const Out h3[3] = {{qo, op(ws + u[0], d, dh), zb[0], zi, d},
                       {qo, op(ws + u[1], d, dh), zb[1], zi, d},
                       {doo, op(ws + u[2], d, dh), zb[2], zi, d}};
    int r = outs(h3, 3, n, (int)h);
    if (r) return r;
    r = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
      return launch_swiglu_apply_rows(zb[0], zb[1], zb[2], zi, pq, T * 2 * h, hq, zi, p.BH, n, (int)h, p.bf16, s);
    });
    if (r) return r;
    return grads(op(pq, 2 * h, T * 2 * h), op(pq + h * esz, 2 * h, T * 2 * h), qo, doo, op(hq, h, zi), apart, n,
                 split_len, &a_ns, into);
  };
  auto dq_out = [&](int64_t a, const uint8_t* bt, int64_t bt_ld) -> Out {
    return Out{op(pq, 2 * h, T * 2 * h), op(bt, bt_ld, d * bt_ld), (uint8_t*)dq + a * d * esz, n_q * d, 2 * h};
  };
  auto pset = [&](float* base, int ns, int m) -> PartSet { return PartSet{base + m * dh, ns, psplit, 3 * dh}; };
  // The running cotangent of the current weights lives in dW; `first` while
  // it still has to start from dW_final (or zero). The partials of the
  // gradient's own dependence on W (bpart) and of an apply (apart) stay
  // pending until the next update's reverse adds them, or a flush does.
  bool first = true;
  bool a_pending = false, b_pending = false;
  auto flush = [&]() -> int {
    if (!first && !a_pending && !b_pending) return LACT_OK;
    for (int m = 0; m < 3; ++m) {
      const PartSet s0 = b_pending ? pset(bpart, b_ns, m) : PartSet{};
      const PartSet s1 = a_pending ? pset(apart, a_ns, m) : PartSet{};
      const int mode = first ? (dWf[m] ? 1 : 0) : 2;
      const int r = timed(LACT_KCLASS_UPDATE, 0.0, s,
                          [&] { return launch_accum(dW[m], dh, dWf[m], dh, mode, s0, s1, p.BH, dh, s); });
      if (r) return r;
    }
    first = a_pending = b_pending = false;
    return LACT_OK;
  };
  for (auto it = segs.rbegin(); it != segs.rend(); ++it) {
    const BSeg& g = *it;
    const int64_t s0 = g.b, n = g.e - g.b;
    if (g.mode == LACT_SEG_APPLY_ONLY) {   // in pieces of up to T rows, with the weights of that time
      if (a_pending) {
        rc = flush();
        if (rc) return rc;
      }
      rc = weight_copies(g.before, L.off_a, bq, 2 * h, nullptr);
      if (rc) return rc;
      for (int64_t a = g.b; a < g.e; a += T) {
        const int64_t na = std::min(T, g.e - a);
        Pending pend;   // the apply's weight cotangents share the dq launch
        rc = apply_back(a, na, L.off_a, L.tail_split, &pend);
        if (rc) return rc;
        const Out o = dq_out(a, bq, 2 * h);
        rc = outs(&o, 1, na, (int)d, &pend);
        if (rc) return rc;
        a_pending = true;
        rc = flush();
        if (rc) return rc;
      }
      continue;
    }
    const int64_t u = g.before;
    const bool then_apply = g.mode == LACT_SEG_UPDATE_THEN_APPLY;
    const bool applies = g.mode != LACT_SEG_UPDATE_ONLY;
    if (then_apply) {   // applied with the weights leaving the update: its cotangent joins first
      if (a_pending) {
        rc = flush();
        if (rc) return rc;
      }
      rc = weight_copies(u + 1, L.off_a, bq, 2 * h, nullptr);
      if (!rc) rc = apply_back(s0, n, L.off_a, p.split_len);
      if (rc) return rc;
      a_pending = true;
    }
    if (first) {   // the update's reverse reads the running cotangent
      const bool ap = a_pending, bp = b_pending;
      a_pending = b_pending = false;
      rc = flush();
      if (rc) return rc;
      a_pending = ap;
      b_pending = bp;
    }
    // the update's reverse: W1, W3 ([h x d]) and W2 ([d x h]) in one launch
    const NsBwd nb{p, L.ns, ws, s, desc->ns_steps, {(int)h, (int)d, (int)h}, {(int)d, (int)h, (int)d}, u};
    float* gslot = reinterpret_cast<float*>(ws + L.off_P + (size_t)u * L.slotP);
    const float* mnext[3] = {mom ? mtraj(u + 1, 0) : nullptr, mom ? mtraj(u + 1, 1) : nullptr,
                             mom ? mtraj(u + 1, 2) : nullptr};
    if (p.muon) {   // the steps are Muon(g_j), or Muon(M_j) with momentum: kept iterates, else a replay
      rc = nb.kept() ? nb.prepare(gslot, p.nsplit, psplit, mom ? mnext : nullptr)
                     : nb.forward(gslot, p.nsplit, psplit, mom ? mnext : nullptr);
      if (rc) return rc;
    }
    VjpArgs va[3] = {};
    for (int m = 0; m < 3; ++m) {
      VjpArgs& x = va[m];
      const bool w2 = m == 1;
      x.W = traj(u, m);
      x.w_inst = dh;
      x.P = p.muon ? pset(nb.pst(), 1, m)
                   : (mom ? PartSet{mnext[m], 1, 0, dh, -1.0f} : pset(gslot, p.nsplit, m));
      if (b_pending) x.pre[0] = pset(bpart, b_ns, m);
      if (a_pending) x.pre[1] = pset(apart, a_ns, m);
      x.G = dW[m];
      x.g_inst = dh;
      if (w2) {   // U2 row-major into [U2 | W2], U2^T for V U2
        x.Ub = bv;
        x.ub_ld = 2 * h;
        x.ub_inst = d * 2 * h;
        x.UT = ur[2];
        x.ut_ld = d;
        x.ut_inst = dh;
      } else {    // U1, U3 row-major for K U^T; transposed into [U3^T | U1^T | ...]
        x.Ub = ur[m == 0 ? 0 : 1];
        x.ub_ld = d;
        x.ub_inst = dh;
        x.UT = bk + (m == 0 ? h : 0) * esz;
        x.ut_ld = 4 * h;
        x.ut_inst = d * 4 * h;
      }
      x.BH = p.BH;
      x.R = (int)(w2 ? d : h);
      x.L = (int)(w2 ? h : d);
      if (p.muon || mom) {   // the update's cotangent in fp32 (Newton-Schulz or momentum reverse next)
        x.Ub = x.UT = nullptr;
        x.U32 = (p.muon ? nb.at<float>(L.ns.ustep) : reinterpret_cast<float*>(ws + L.off_mu)) + m * dh;
        x.u32_inst = 3 * dh;
      }
    }
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_vjp(va, 3, p.bf16, s); });
    if (rc) return rc;
    if (p.muon) {
      rc = nb.reverse();
      if (rc) return rc;
    }
    if (mom) {   // dM' = carried - (step's share); the gradient's cotangent; carry bbar dM'; dbeta
      MomBwdArgs ma{};
      ma.U = p.muon ? nb.at<float>(L.ns.ug) : reinterpret_cast<float*>(ws + L.off_mu);
      for (int m = 0; m < 3; ++m) {
        ma.R[m] = dMo[m];
        ma.M[m] = mtraj(u, m);
      }
      ma.bbar = bbar_all + u;
      ma.bbar_inst = nupd;
      ma.part = reinterpret_cast<float*>(ws + L.off_mpart);
      ma.BH = p.BH;
      ma.nmat = 3;
      ma.nblk = kMomBlocks;
      ma.dh = dh;
      rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_mom_bwd(ma, s); });
      if (!rc) rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] {
        return launch_mom_dbeta(ma.part, kMomBlocks, p.BH, dbeta + s0, n_kv, n, s);
      });
      if (rc) return rc;
    }
    if (p.muon || mom) {   // the gradients' cotangents (negated) into the operand layouts
      const float* ug = p.muon ? nb.at<float>(L.ns.ug) : reinterpret_cast<float*>(ws + L.off_mu);
      const CopySeg cs[3] = {{ug, 3 * dh, (int)h, (int)d, ur[0], d, dh, bk + h * esz, 4 * h, d * 4 * h},
                             {ug + 2 * dh, 3 * dh, (int)h, (int)d, ur[1], d, dh, bk, 4 * h, d * 4 * h},
                             {ug + dh, 3 * dh, (int)d, (int)h, bv, 2 * h, d * 2 * h, ur[2], d, dh}};
      rc = timed(LACT_KCLASS_NS, 0.0, s, [&] { return launch_copies(cs, 3, p.BH, p.bf16, s); });
      if (rc) return rc;
    }
    a_pending = b_pending = false;
    rc = weight_copies(u, L.off_u, bk + 2 * h * esz, 4 * h, bv + h * esz);
    if (rc) return rc;
    const Operand ko = op(kb + s0 * d * esz, d, n_kv * d), vo = op(vb + s0 * d * esz, d, n_kv * d);
    // Z1 = K W1^T, Z3 = K W3^T and C = V W2 of this update: kept by its replay
    uint8_t* kz = ws + L.off_keep + (size_t)u * L.keep_slot;
    const size_t kzm = (size_t)p.BH * p.C * h * esz;
    const Out x3[3] = {{ko, op(ur[0], d, dh), zb[3], zi, d},
                       {ko, op(ur[1], d, dh), zb[4], zi, d},
                       {vo, op(ur[2], d, dh), zb[5], zi, d}};
    rc = outs(x3, 3, n, (int)h);
    if (rc) return rc;
    SwigluRowsArgs ra{};
    ra.Z1 = kz;
    ra.Z3 = kz + kzm;
    ra.C = kz + 2 * kzm;
    ra.z_inst = p.C * h;
    ra.X1 = zb[3];
    ra.X3 = zb[4];
    ra.Y2 = zb[5];
    ra.in_inst = zi;
    ra.eta = eta + s0 * p.es;
    ra.eta_inst = n_kv;
    ra.eta_cols = p.es;
    ra.Pk = pk;
    ra.pk_inst = T * 4 * h;
    ra.Pv = pv;
    ra.pv_inst = T * 2 * h;
    ra.deta = deta + s0 * p.es;
    ra.BH = p.BH;
    ra.n = n;
    ra.h = (int)h;
    rc = timed(LACT_KCLASS_UPDATE, 0.0, s, [&] { return launch_swiglu_rows(ra, p.bf16, s); });
    if (rc) return rc;
    // One launch: the weight cotangents of the apply with the entering
    // weights (apart) and of the gradient's own dependence on W (bpart), then
    // dk (a sum over 4h), dv and dq (over 2h). The five products read
    // buffers that are complete by now and write disjoint ones.
    Pending pend;
    if (applies && !then_apply) {   // applied with the weights entering the update (their copies are in place)
      rc = apply_back(s0, n, L.off_u, p.split_len, &pend);
      if (rc) return rc;
    }
    rc = grads(op(pk + 2 * h * esz, 4 * h, T * 4 * h), op(pk + 3 * h * esz, 4 * h, T * 4 * h), ko, vo,
               op(pv + h * esz, 2 * h, T * 2 * h), bpart, n, p.split_len, &b_ns, &pend);
    if (rc) return rc;
    const Out kvq[3] = {
        {op(pk, 4 * h, T * 4 * h), op(bk, 4 * h, d * 4 * h), (uint8_t*)dk + s0 * d * esz, n_kv * d, 4 * h},
        {op(pv, 2 * h, T * 2 * h), op(bv, 2 * h, d * 2 * h), (uint8_t*)dv + s0 * d * esz, n_kv * d, 2 * h},
        then_apply ? dq_out(s0, bq, 2 * h) : dq_out(s0, bk + 2 * h * esz, 4 * h)};
    rc = outs(kvq, applies ? 3 : 2, n, (int)d, &pend);
    if (rc) return rc;
    b_pending = true;
    a_pending = applies && !then_apply;   // the entering weights' apply joins before the previous update's reverse
  }
  return flush();
}

}  // namespace
}  // namespace lact

using namespace lact;

extern "C" {

int lact_check_desc(const lact_desc* desc) { return check_desc(desc); }

size_t lact_workspace_bytes(const lact_desc* desc, int* err) {
  const int rc = check_desc(desc);
  if (err) *err = rc;
  if (rc) return 0;
  return make_plan(desc).total;
}

int lact_forward(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                 float* W1, float* W2, float* W3, void* o, void* workspace, size_t workspace_bytes,
                 void* stream) {
  return run_forward(desc, q, k, v, eta, nullptr, W1, W2, W3, nullptr, o, workspace, workspace_bytes,
                     stream);
}

size_t lact_backward_workspace_bytes(const lact_desc* desc, int* err) {
  int rc = check_desc(desc);
  size_t total = 0;
  if (!rc && desc->fast_weight == LACT_FW_LINEAR) {
    BwdLayout L;
    rc = bwd_layout(desc, &L);
    total = L.total;
  } else if (!rc) {
    SwBwdLayout L;
    rc = sw_bwd_layout(desc, &L);
    total = L.total;
  }
  if (err) *err = rc;
  return rc ? 0 : total;
}

size_t lact_backward_momentum_workspace_bytes(const lact_desc* desc, int* err) {
  int rc = check_desc(desc);
  size_t total = 0;
  if (!rc && desc->fast_weight == LACT_FW_LINEAR) {
    BwdLayout L;
    rc = bwd_layout(desc, &L, true);
    total = L.total;
  } else if (!rc) {
    SwBwdLayout L;
    rc = sw_bwd_layout(desc, &L, true);
    total = L.total;
  }
  if (err) *err = rc;
  return rc ? 0 : total;
}

int lact_backward_momentum(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                           const float* beta, const float* W1, const float* W2, const float* W3, const float* M1,
                           const float* M2, const float* M3, const void* dout, const float* dW1_final,
                           const float* dW2_final, const float* dW3_final, const float* dM1_final,
                           const float* dM2_final, const float* dM3_final, void* dq, void* dk, void* dv,
                           float* deta, float* dbeta, float* dW1, float* dW2, float* dW3, float* dM1, float* dM2,
                           float* dM3, void* workspace, size_t workspace_bytes, void* stream) {
  const int rc = check_desc(desc);
  if (rc) return rc;
  if (!M1 || !dM1) return LACT_EINVAL;   // the entry point's state and its cotangent
  if (desc->fast_weight == LACT_FW_LINEAR)
    return run_backward_linear(desc, q, k, v, eta, W1, dout, dW1_final, dq, dk, dv, deta, dW1, workspace,
                               workspace_bytes, stream, beta, M1, dM1_final, dbeta, dM1);
  const float* W0[3] = {W1, W2, W3};
  const float* dWf[3] = {dW1_final, dW2_final, dW3_final};
  float* const dW[3] = {dW1, dW2, dW3};
  const float* M0[3] = {M1, M2, M3};
  const float* dMf[3] = {dM1_final, dM2_final, dM3_final};
  float* const dMo[3] = {dM1, dM2, dM3};
  return run_backward_swiglu(desc, q, k, v, eta, W0, dout, dWf, dq, dk, dv, deta, dW, workspace, workspace_bytes,
                             stream, beta, M0, dMf, dbeta, dMo);
}

size_t lact_backward_schedule_workspace_bytes(const lact_desc* desc, const lact_segment* segs, int64_t nseg,
                                              int momentum, int* err) {
  int rc = check_desc(desc);
  std::vector<BSeg> bs;
  int64_t nupd = 0, longest = 0;
  if (!rc && nseg < 0) rc = LACT_EINVAL;
  if (!rc) rc = backward_segments(desc, segs, nseg, &bs, &nupd, &longest);
  size_t total = 0;
  if (!rc && desc->fast_weight == LACT_FW_LINEAR) {
    BwdLayout L;
    rc = bwd_layout(desc, &L, momentum != 0, nupd, longest);
    total = L.total;
  } else if (!rc) {
    SwBwdLayout L;
    rc = sw_bwd_layout(desc, &L, momentum != 0, nupd, longest);
    total = L.total;
  }
  if (err) *err = rc;
  return rc ? 0 : total;
}

int lact_backward_schedule(const lact_desc* desc, const lact_segment* segs, int64_t nseg, const void* q,
                           const void* k, const void* v, const float* eta, const float* beta, const float* W1,
                           const float* W2, const float* W3, const float* M1, const float* M2, const float* M3,
                           const void* dout, const float* dW1_final, const float* dW2_final, const float* dW3_final,
                           const float* dM1_final, const float* dM2_final, const float* dM3_final, void* dq,
                           void* dk, void* dv, float* deta, float* dbeta, float* dW1, float* dW2, float* dW3,
                           float* dM1, float* dM2, float* dM3, void* workspace, size_t workspace_bytes,
                           void* stream) {
  const int rc = check_desc(desc);
  if (rc) return rc;
  if (nseg < 0 || (nseg > 0 && !segs)) return LACT_EINVAL;
  const bool mom = M1 != nullptr;
  if (desc->fast_weight == LACT_FW_LINEAR)
    return run_backward_linear(desc, q, k, v, eta, W1, dout, dW1_final, dq, dk, dv, deta, dW1, workspace,
                               workspace_bytes, stream, mom ? beta : nullptr, M1, mom ? dM1_final : nullptr,
                               mom ? dbeta : nullptr, mom ? dM1 : nullptr, segs, nseg);
  const float* W0[3] = {W1, W2, W3};
  const float* dWf[3] = {dW1_final, dW2_final, dW3_final};
  float* const dW[3] = {dW1, dW2, dW3};
  const float* M0[3] = {M1, M2, M3};
  const float* dMf[3] = {dM1_final, dM2_final, dM3_final};
  float* const dMo[3] = {dM1, dM2, dM3};
  return run_backward_swiglu(desc, q, k, v, eta, W0, dout, dWf, dq, dk, dv, deta, dW, workspace, workspace_bytes,
                             stream, mom ? beta : nullptr, mom ? M0 : nullptr, mom ? dMf : nullptr,
                             mom ? dbeta : nullptr, mom ? dMo : nullptr, segs, nseg);
}

int lact_backward(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                  const float* W1, const float* W2, const float* W3, const void* dout, const float* dW1_final,
                  const float* dW2_final, const float* dW3_final, void* dq, void* dk, void* dv, float* deta,
                  float* dW1, float* dW2, float* dW3, void* workspace, size_t workspace_bytes, void* stream) {
  const float* W0[3] = {W1, W2, W3};
  const float* dWf[3] = {dW1_final, dW2_final, dW3_final};
  float* const dW[3] = {dW1, dW2, dW3};
  return run_backward_swiglu(desc, q, k, v, eta, W0, dout, dWf, dq, dk, dv, deta, dW, workspace, workspace_bytes,
                             stream);
}

int lact_backward_linear(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                         const float* W0, const void* dout, const float* dW_final, void* dq, void* dk, void* dv,
                         float* deta, float* dW0, void* workspace, size_t workspace_bytes, void* stream) {
  return run_backward_linear(desc, q, k, v, eta, W0, dout, dW_final, dq, dk, dv, deta, dW0, workspace,
                             workspace_bytes, stream);
}

int lact_forward_noalloc(const lact_desc* desc, const void* q, const void* k, const void* v, const float* eta,
                         float* W1, float* W2, float* W3, void* o, void* stream) {
  return run_forward(desc, q, k, v, eta, nullptr, W1, W2, W3, nullptr, o, nullptr, 0, stream, true);
}

int lact_prologue(const lact_desc* desc, const void* qkv, const float* lr_raw, float lr_bias, const float* beta_raw,
                  void* q, void* k, void* v, float* eta, float* beta, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  const bool any_q = desc->n_q > 0, any_kv = desc->n_kv > 0;
  if (any_q && (!qkv || !q || !lr_raw)) return LACT_EINVAL;
  if (any_kv && (!k || !v || !eta)) return LACT_EINVAL;
  if ((beta_raw == nullptr) != (beta == nullptr)) return LACT_EINVAL;
  if (!(lr_bias == lr_bias) || lr_bias - lr_bias != 0.0f) return LACT_EINVAL;   // finite
  if (any_q && (misaligned(qkv) || misaligned(q) || ((uintptr_t)lr_raw & 3))) return LACT_EALIGN;
  if (any_kv && (misaligned(k) || misaligned(v) || ((uintptr_t)eta & 3))) return LACT_EALIGN;
  if (beta && (((uintptr_t)beta & 3) || ((uintptr_t)beta_raw & 3))) return LACT_EALIGN;
  PrologueArgs a{};
  a.qkv = qkv;
  a.lr_raw = lr_raw;
  a.beta_raw = beta_raw;
  a.lr_bias = lr_bias;
  a.q = q;
  a.k = k;
  a.v = v;
  a.eta = eta;
  a.beta = beta;
  a.B = desc->B;
  a.H = desc->H;
  a.hd = desc->d;
  a.R = desc->eta_per_matrix ? 3 : 1;
  a.L = desc->n_q;
  a.n_kv = desc->n_kv;
  const bool bf16 = desc->io_dtype == LACT_IO_BF16;
  hipStream_t s = (hipStream_t)stream;
  return timed(LACT_KCLASS_IO, 0.0, s, [&] { return launch_prologue(a, bf16, s); });
}

int lact_rmsnorm_out(const lact_desc* desc, const void* o, const float* weight, float eps, void* y, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  if (!(eps >= 0.0f) || eps - eps != 0.0f) return LACT_EINVAL;   // finite, >= 0
  if (desc->n_q > 0 && (!o || !y)) return LACT_EINVAL;
  if (desc->n_q > 0 && (misaligned(o) || misaligned(y))) return LACT_EALIGN;
  if (weight && ((uintptr_t)weight & 3)) return LACT_EALIGN;
  RmsArgs a{};
  a.o = o;
  a.weight = weight;
  a.y = y;
  a.eps = eps;
  a.B = desc->B;
  a.H = desc->H;
  a.hd = desc->d;
  a.L = desc->n_q;
  const bool bf16 = desc->io_dtype == LACT_IO_BF16;
  hipStream_t s = (hipStream_t)stream;
  return timed(LACT_KCLASS_IO, 0.0, s, [&] { return launch_rmsnorm_out(a, bf16, s); });
}

int lact_prologue_backward(const lact_desc* desc, const void* qkv, const float* lr_raw, float lr_bias,
                           const float* beta_raw, const void* dq, const void* dk, const void* dv, const float* deta,
                           const float* dbeta, void* dqkv, float* dlr_raw, float* dbeta_raw, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  const bool any_q = desc->n_q > 0, any_kv = desc->n_kv > 0;
  if (any_q && (!qkv || !lr_raw || !dq || !dqkv || !dlr_raw)) return LACT_EINVAL;
  if (any_kv && (!dk || !dv || !deta)) return LACT_EINVAL;
  // the momentum logits' cotangent: beta_raw, dbeta and dbeta_raw together, or none
  if ((beta_raw == nullptr) != (dbeta_raw == nullptr) || (dbeta_raw && any_kv && !dbeta)) return LACT_EINVAL;
  if (!(lr_bias == lr_bias) || lr_bias - lr_bias != 0.0f) return LACT_EINVAL;   // finite
  if (any_q && (misaligned(qkv) || misaligned(dq) || misaligned(dqkv) || ((uintptr_t)lr_raw & 3) ||
                ((uintptr_t)dlr_raw & 3)))
    return LACT_EALIGN;
  if (any_kv && (misaligned(dk) || misaligned(dv) || ((uintptr_t)deta & 3))) return LACT_EALIGN;
  if (dbeta_raw && (((uintptr_t)beta_raw & 3) || ((uintptr_t)dbeta_raw & 3) || ((uintptr_t)dbeta & 3)))
    return LACT_EALIGN;
  PrologueBwdArgs a{};
  a.qkv = qkv;
  a.lr_raw = lr_raw;
  a.beta_raw = beta_raw;
  a.lr_bias = lr_bias;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.deta = deta;
  a.dbeta = dbeta;
  a.dqkv = dqkv;
  a.dlr_raw = dlr_raw;
  a.dbeta_raw = dbeta_raw;
  a.B = desc->B;
  a.H = desc->H;
  a.hd = desc->d;
  a.R = desc->eta_per_matrix ? 3 : 1;
  a.L = desc->n_q;
  a.n_kv = desc->n_kv;
  const bool bf16 = desc->io_dtype == LACT_IO_BF16;
  hipStream_t s = (hipStream_t)stream;
  return timed(LACT_KCLASS_IO, 0.0, s, [&] { return launch_prologue_bwd(a, bf16, s); });
}

size_t lact_rmsnorm_out_backward_workspace_bytes(const lact_desc* desc, int with_weight, int* err) {
  const int rc = check_desc(desc);
  if (err) *err = rc;
  if (rc) return 0;
  if (!with_weight) return 0;
  const size_t r = align_up((size_t)desc->B * desc->n_q * desc->H * 4);
  const size_t part = (size_t)rms_dw_splits(desc->B, desc->n_q, desc->H, desc->d) * desc->H * desc->d * 4;
  return align_up(r + part);
}

int lact_rmsnorm_out_backward(const lact_desc* desc, const void* o, const float* weight, float eps, const void* dy,
                              void* d_o, float* dweight, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  if (!(eps >= 0.0f) || eps - eps != 0.0f) return LACT_EINVAL;   // finite, >= 0
  if (desc->n_q > 0 && (!o || !dy || !d_o)) return LACT_EINVAL;
  if (dweight && !weight) return LACT_EINVAL;
  if (desc->n_q > 0 && (misaligned(o) || misaligned(dy) || misaligned(d_o))) return LACT_EALIGN;
  if ((weight && ((uintptr_t)weight & 3)) || (dweight && ((uintptr_t)dweight & 3))) return LACT_EALIGN;
  const size_t need = lact_rmsnorm_out_backward_workspace_bytes(desc, dweight != nullptr, nullptr);
  if (need && (!workspace || workspace_bytes < need)) return LACT_EWORKSPACE;
  if (need && ((uintptr_t)workspace & (kAlign - 1))) return LACT_EALIGN;
  RmsBwdArgs a{};
  a.o = o;
  a.weight = weight;
  a.dy = dy;
  a.d_o = d_o;
  a.dweight = dweight;
  a.r = dweight ? reinterpret_cast<float*>(workspace) : nullptr;
  a.part = dweight ? reinterpret_cast<float*>((uint8_t*)workspace +
                                              align_up((size_t)desc->B * desc->n_q * desc->H * 4))
                   : nullptr;
  a.eps = eps;
  a.B = desc->B;
  a.H = desc->H;
  a.hd = desc->d;
  a.L = desc->n_q;
  const bool bf16 = desc->io_dtype == LACT_IO_BF16;
  hipStream_t s = (hipStream_t)stream;
  if (dweight && desc->n_q == 0) {   // no tokens: a zero cotangent
    return timed(LACT_KCLASS_IO, 0.0, s, [&] {
      return launch_zero_f32(dweight, 1, 0, 0, (int64_t)desc->H * desc->d, s);
    });
  }
  return timed(LACT_KCLASS_IO, 0.0, s, [&] { return launch_rmsnorm_out_bwd(a, bf16, s); });
}

int lact_forward_schedule(const lact_desc* desc, const lact_segment* segs, int64_t nseg, const void* q,
                          const void* k, const void* v, const float* eta, const float* beta, float* W1, float* W2,
                          float* W3, float* M1, float* M2, float* M3, void* o, void* workspace,
                          size_t workspace_bytes, void* stream) {
  float* const M[3] = {M1, M2, M3};
  return run_schedule(desc, segs, nseg, q, k, v, eta, beta, W1, W2, W3, M1 ? M : nullptr, o, workspace,
                      workspace_bytes, stream);
}

int lact_forward_momentum(const lact_desc* desc, const void* q, const void* k, const void* v,
                          const float* eta, const float* beta, float* W1, float* W2, float* W3, float* M1,
                          float* M2, float* M3, void* o, void* workspace, size_t workspace_bytes,
                          void* stream) {
  float* const M[3] = {M1, M2, M3};
  return run_forward(desc, q, k, v, eta, beta, W1, W2, W3, M, o, workspace, workspace_bytes, stream);
}

int lact_timing_enable(int enable) {
  g_timing.enabled = enable != 0;
  return LACT_OK;
}

int lact_timing_reset(void) {
  for (auto& t : g_timing.pending) {
    g_timing.pool.push_back(t.a);
    g_timing.pool.push_back(t.b);
  }
  g_timing.pending.clear();
  for (int i = 0; i < LACT_KCLASS_COUNT; ++i) {
    g_timing.launches[i] = 0;
    g_timing.ms[i] = 0;
    g_timing.flops[i] = 0;
  }
  return LACT_OK;
}

int lact_timing_read(int kclass, int64_t* launches, double* total_ms, double* flops) {
  if (kclass < 0 || kclass >= LACT_KCLASS_COUNT) return LACT_EINVAL;
  // Fold every recorded launch into the totals.
  for (auto& t : g_timing.pending) {
    if (hipEventSynchronize(t.b) != hipSuccess) return record_hip(hipGetLastError());
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.a, t.b) != hipSuccess) return record_hip(hipGetLastError());
    g_timing.launches[t.kclass] += 1;
    g_timing.ms[t.kclass] += ms;
    g_timing.flops[t.kclass] += t.flops;
    g_timing.pool.push_back(t.a);
    g_timing.pool.push_back(t.b);
  }
  g_timing.pending.clear();
  if (launches) *launches = g_timing.launches[kclass];
  if (total_ms) *total_ms = g_timing.ms[kclass];
  if (flops) *flops = g_timing.flops[kclass];
  return LACT_OK;
}

const char* lact_strerror(int code) {
  switch (code) {
    case LACT_OK: return "ok";
    case LACT_EINVAL: return "invalid argument";
    case LACT_EALIGN: return "pointer not 16-byte aligned (workspace: 256-byte)";
    case LACT_EWORKSPACE: return "workspace missing or too small";
    case LACT_EUNSUPPORTED: return "shape or option outside the kernels' envelope";
    case LACT_EHIP: return "HIP runtime error (see lact_last_hip_error)";
    case LACT_ESCRATCH: return "the call needs more scratch memory than the fixed per-device array of "
                               "lact_forward_noalloc holds (LACT_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown error";
  }
}

const char* lact_last_hip_error(void) { return g_hip_err; }

const char* lact_version(void) { return "lact-gfx950 0.1.0"; }

}  // extern "C"
