// C ABI of the DendSN layer scan: argument checks, launch planning, dispatch,
// and the deterministic parameter-gradient finalize kernel.
#include <math.h>
#include <string.h>

#include <mutex>
#include <string>

#include "dendsn.h"
#include "dendsn_kernels.h"

namespace dendsn {

hipError_t launch_fwd_f32(const Plan& pl, const FwdArgs& fa, int psi, hipStream_t stream);
hipError_t launch_fwd_bf16(const Plan& pl, const FwdArgs& fa, int psi, hipStream_t stream);
hipError_t launch_bwd_f32_sg0(const Plan& pl, const BwdArgs& ba, int psi, hipStream_t stream);
hipError_t launch_bwd_f32_sg1(const Plan& pl, const BwdArgs& ba, int psi, hipStream_t stream);
hipError_t launch_bwd_bf16_sg0(const Plan& pl, const BwdArgs& ba, int psi, hipStream_t stream);
hipError_t launch_bwd_bf16_sg1(const Plan& pl, const BwdArgs& ba, int psi, hipStream_t stream);
hipError_t launch_fwd_f32_kc(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream);
hipError_t launch_fwd_bf16_kc(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream);
hipError_t launch_bwd_f32_kc_sg0(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_bwd_f32_kc_sg1(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_bwd_bf16_kc_sg0(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_bwd_bf16_kc_sg1(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_fwd_f32_cm(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream);
hipError_t launch_fwd_bf16_cm(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream);
hipError_t launch_bwd_f32_cm_sg0(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_bwd_f32_cm_sg1(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_bwd_bf16_cm_sg0(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);
hipError_t launch_bwd_bf16_cm_sg1(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream);

// Fixed-order float64 sums of the per-block partials into the parameter
// gradients.  Outputs o = c * W + ol with W = 2 B + P: ol < B is g_kappa of
// branch ol, then g_xi of the P compartments, then g_zeta of the B branches.
// Blocks 0 and 1 reduce the g_alpha and g_beta partials (first, so that their
// longer serial sums overlap the rest).
__global__ void __launch_bounds__(kThreads) dendsn_finalize_kernel(FinArgs f) {
  const int tid = threadIdx.x;
  const int W = 2 * f.B + f.P;
  const int64_t nout = f.C * W;
  if (blockIdx.x < 2) {  // block 0: g_alpha; block 1: g_beta
    const bool is_alpha = blockIdx.x == 0;
    const float* src = is_alpha ? f.wsA : f.wsB;
    __shared__ double sh[kThreads];
    // A thread sums src[tid], src[tid + 256], ... in that order.  Eight loads
    // are issued together, unconditionally (an index past the end reads the
    // last element again and its term is dropped), so they share one round trip.
    constexpr int U = 8;
    const int64_t last = f.nA - 1;
    double s = 0.0;
    for (int64_t i0 = tid; i0 < f.nA; i0 += int64_t(U) * kThreads) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = src[min(i0 + int64_t(u) * kThreads, last)];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (i0 + int64_t(u) * kThreads <= last) s += double(v[u]);
    }
    sh[tid] = s;
    __syncthreads();
    for (int w = kThreads / 2; w >= 1; w >>= 1) {
      if (tid < w) sh[tid] += sh[tid + w];
      __syncthreads();
    }
    if (tid == 0) {
      if (is_alpha && f.ga) f.ga[0] = f.stateful ? float(sh[0]) : 0.0f;
      if (!is_alpha && f.gb) f.gb[0] = float(sh[0]);
    }
    return;
  }
  const bool wide = f.wide != 0;
  const int lane = tid & 63;
  const int64_t o = wide ? int64_t(blockIdx.x - 2) * (kThreads / 64) + (tid >> 6)
                         : int64_t(blockIdx.x - 2) * kThreads + tid;
  if (!wide && o >= nout) return;  // (wide: every lane stays for the shuffles)
  // Where the output goes, worked out first so that its branch's gate is read
  // in the same round trip as the partial sums.
  const int64_t oq = o < nout ? o : nout - 1;
  const int64_t c = oq / W;
  const int ol = int(oq % W);
  float* out;
  int64_t idx;
  int b;  // the branch the output belongs to
  if (ol < f.B) {
    out = f.gk; idx = c * f.B + ol; b = ol;
  } else if (ol < f.B + f.P) {
    out = f.gxi; idx = c * f.P + (ol - f.B); b = (ol - f.B) / f.KC;
  } else {
    out = f.gz; idx = c * f.B + (ol - f.B - f.P); b = ol - f.B - f.P;
  }
  const uint8_t* gate = f.mask ? f.mask + c * f.B + b : nullptr;
  bool on = true;
  double s = 0.0;
  if (wide) {  // one wave per output, lanes stride over its contiguous slots
    if (o < nout)
      for (int64_t p = lane; p < f.slots; p += 64) s += double(f.wsP[o * f.slots + p]);
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
    if (lane != 0 || o >= nout) return;
    if (gate) on = *gate != 0;
  } else {     // one thread per output, slots in order
    // slots in groups of four, each group's loads issued together (a slot past
    // the last reads the last one again and its term is dropped); the gate is
    // read behind the first group's loads
    const int64_t last = f.slots - 1;
    for (int64_t p0 = 0; p0 <= last; p0 += 4) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = f.wsP[min(p0 + u, last) * nout + o];
      if (p0 == 0 && gate) on = *gate != 0;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (p0 + u <= last) s += double(v[u]);
    }
  }
  if (!out) return;
  out[idx] = on ? float(s) : 0.0f;
}

}  // namespace dendsn

using namespace dendsn;

namespace {

thread_local std::string g_last_error;

dendsn_status fail(dendsn_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// (BL, L) for KC compartments per branch.  KC = 1: a vector-width lane split
// when the branch count allows one (16 bytes per lane; the bf16 backward takes
// 8 bytes, 4 branches, per lane from 16 up to 64 branches: measured 10 % faster
// than 8 branches per lane, whose stash fills the registers; with 8 branches
// one lane of 8 is 3 % faster than two lanes of 4, half the soma work per
// branch), else a generic split with up to 8 branches per lane over 1 or 2 lanes.  KC = 2 or 4: 16 bytes of compartments per lane
// (BL KC = 4 for fp32, 8 for bf16) when the branch count allows, else one lane
// holds the whole neuron (B KC <= 14).
bool choose_mapping(int B, int KC, int io, bool bwd, int* BL, int* L, int* fast) {
  if (KC == 1) {
    // The fp32 forward of 16 branches: 8 per lane over two lanes (the same
    // balanced branch-sum tree as the backward's 4 over four).  Measured on
    // MI355X, 64-step fully connected layer: 122 -> 117-120 us (each wave reads
    // 2 KiB of a row instead of 1 KiB, half the waves); with 32 branches (8 over
    // four lanes) the gated layer's forward was 2 % slower, with one lane of 16
    // the 16-branch forward 35 % slower.
    if (!bwd && io == DENDSN_IO_F32 && B == 16) {
      *BL = 8; *L = 2; *fast = 1;
      return true;
    }
    const int blv = (io == DENDSN_IO_BF16 && B % 8 == 0 && !(bwd && B > 8 && B <= 64)) ? 8 : 4;
    if (B % blv == 0 && is_pow2(B / blv) && B / blv <= 16) {
      *BL = blv; *L = B / blv; *fast = 1;
      return true;
    }
    for (int l = 1; l <= 2; l *= 2) {
      if (B % l == 0 && B / l <= 8) {
        *BL = B / l; *L = l; *fast = 0;
        return true;
      }
    }
    return false;
  }
  if (KC != 2 && KC != 4) return false;
  const int blv = (io == DENDSN_IO_BF16 ? 8 : 4) / KC;
  if (B % blv == 0 && is_pow2(B / blv) && B / blv <= 16) {
    *BL = blv; *L = B / blv; *fast = 1;
    return true;
  }
  if ((KC == 2 && B <= 7 && B != 4) || (KC == 4 && B <= 3)) {
    *BL = B; *L = 1; *fast = 0;
    return true;
  }
  return false;
}

// The channel-major layout (S > 1; with S = 1 it is the same memory as
// [T, N, P]): the fewest lanes per neuron (a power of two dividing B) that leave
// at most 4 compartments in a lane, if a compiled mapping has it.
bool channel_major(const dendsn_cfg* c) { return c->layout == DENDSN_LAYOUT_CHANNEL_MAJOR && c->S > 1; }

bool cm_mapping(int B, int KC, int* BL, int* L) {
  int l = 1;
  while ((B * KC) / l > 4 && B % (2 * l) == 0 && 2 * l <= 16) l *= 2;
  const int bl = B / l;
#define DENDSN_IN(BL_, L_, KC_) \
  if (bl == BL_ && l == L_ && KC == KC_) { *BL = bl; *L = l; return true; }
  DENDSN_CM(DENDSN_IN)
#undef DENDSN_IN
  return false;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// No neuron-step at all (T = 0 or N = 0): the forward has nothing to compute
// and the backward's parameter gradients are empty sums, +0.
bool empty_layer(const dendsn_cfg* c) { return c->T == 0 || c->batch == 0 || c->C == 0 || c->S == 0; }

// Workspace of an empty layer: nothing is read or written there, but the size
// stays positive like every other layer's.
constexpr size_t kEmptyWorkspace = 256;

dendsn_status check_cfg(const dendsn_cfg* c) {
  if (!c) return fail(DENDSN_E_INVALID, "cfg is NULL");
  // Zero steps, samples, channels or positions make an empty layer (valid).
  if (c->T < 0 || c->T > INT32_MAX) return fail(DENDSN_E_INVALID, "T must be in [0, 2^31)");
  if (c->batch < 0) return fail(DENDSN_E_INVALID, "batch must be >= 0");
  if (c->C < 0) return fail(DENDSN_E_INVALID, "C must be >= 0");
  if (c->S < 0) return fail(DENDSN_E_INVALID, "S must be >= 0");
  if (c->B < 1 || c->B > 128) return fail(DENDSN_E_INVALID, "B must be in [1, 128]");
  if (c->comps_per_branch < 1) return fail(DENDSN_E_INVALID, "comps_per_branch must be >= 1");
  if (c->comps_per_branch != 1 && c->comps_per_branch != 2 && c->comps_per_branch != 4)
    return fail(DENDSN_E_UNSUPPORTED, "comps_per_branch must be 1, 2 or 4");
  if (c->stateful != 0 && c->stateful != 1) return fail(DENDSN_E_INVALID, "stateful must be 0 or 1");
  if (c->detach_reset != 0 && c->detach_reset != 1)
    return fail(DENDSN_E_INVALID, "detach_reset must be 0 or 1");
  if (c->ckpt_every < 1) return fail(DENDSN_E_INVALID, "ckpt_every must be >= 1");
  if (c->io != DENDSN_IO_F32 && c->io != DENDSN_IO_BF16) return fail(DENDSN_E_INVALID, "bad io");
  if (c->psi != DENDSN_PSI_IDENTITY && c->psi != DENDSN_PSI_MEXHAT) return fail(DENDSN_E_INVALID, "bad psi");
  if (c->sg != DENDSN_SG_ATAN && c->sg != DENDSN_SG_SIGMOID) return fail(DENDSN_E_INVALID, "bad sg");
  if (c->sg == DENDSN_SG_SIGMOID && !(isfinite(c->sg_scale) && c->sg_scale > 0.0f))
    return fail(DENDSN_E_INVALID, "sg_scale must be finite and > 0");
  if (!isfinite(c->beta)) return fail(DENDSN_E_INVALID, "beta must be finite");
  if (!isfinite(c->v_th)) return fail(DENDSN_E_INVALID, "v_th must be finite");
  if (c->batch_groups < 0) return fail(DENDSN_E_INVALID, "batch_groups must be >= 0");
  if (c->residual != 0 && c->residual != 1) return fail(DENDSN_E_INVALID, "residual must be 0 or 1");
  if (c->layout != DENDSN_LAYOUT_NPB && c->layout != DENDSN_LAYOUT_CHANNEL_MAJOR)
    return fail(DENDSN_E_INVALID, "bad layout");
  // N and T * N * B must fit comfortably in int64 element counts.
  const int64_t lim = int64_t(1) << 46;
  if (c->C > lim || c->S > lim) return fail(DENDSN_E_INVALID, "C or S too large");
  if (c->C > 0 && c->S > 0 && (c->batch > lim / c->C || c->batch * c->C > lim / c->S))
    return fail(DENDSN_E_INVALID, "N too large");
  const int64_t N = c->batch * c->C * c->S;
  const int64_t P = int64_t(c->B) * c->comps_per_branch;
  if (c->T > 0 && N > (lim / P) / c->T) return fail(DENDSN_E_INVALID, "T * N * P too large");
  int BL, L, fast;
  if (channel_major(c)) {
    if (!cm_mapping(c->B, c->comps_per_branch, &BL, &L))
      return fail(DENDSN_E_UNSUPPORTED, "branch count not covered by the compiled channel-major kernels");
  } else if (!choose_mapping(c->B, c->comps_per_branch, c->io, false, &BL, &L, &fast) ||
             !choose_mapping(c->B, c->comps_per_branch, c->io, true, &BL, &L, &fast)) {
    return fail(DENDSN_E_UNSUPPORTED, "branch count not covered by the compiled kernels");
  }
  return DENDSN_OK;
}

// Tiling and batch grouping.  The two directions may split a neuron over lanes
// differently only where the branch sum's tree stays the same (powers of two),
// so the backward's recompute adds the branch terms as the forward did.
Plan make_plan(const dendsn_cfg* c, bool bwd) {
  Plan p;
  memset(&p, 0, sizeof(p));
  p.KC = c->comps_per_branch;
  if (channel_major(c)) {
    p.cm = 1; p.fast = 0;
    cm_mapping(c->B, c->comps_per_branch, &p.BL, &p.L);
    // Forward: half the lanes when the backward's split is a power of two with at
    // most 4 compartments per lane (measured on MI355X: cifar-shaped B = 8,
    // 523 -> 408 us with one lane and two positions per lane)
    if (!bwd && is_pow2(p.BL) && p.L >= 2 && p.BL * p.KC <= 4) { p.BL *= 2; p.L /= 2; }
  } else {
    choose_mapping(c->B, c->comps_per_branch, c->io, bwd, &p.BL, &p.L, &p.fast);
  }
  const int L = p.L;
  const int esz = c->io == DENDSN_IO_BF16 ? 2 : 4;
  p.nw = 1;
  if (c->S >= kThreads / L) {
    p.mode = kSpatial; p.ways = 1; p.pb = kThreads / L;
    // A lane may take nw positions per batch item, so a wave reads and writes
    // nw x 64 / L adjacent positions per row (fewer, longer-lived waves).
    // Measured on MI355X.  Backward (four steps, 16-byte lane rows): nw = 4 when
    // a neuron spans 2 or 4 lanes (cifar 911 -> 800 us against nw = 2, B = 16
    // 885 -> 810 us; nw = 8 is slower again), nw = 2 with one lane per neuron
    // (3-9 % faster than 1; 4 no better); the channel-major layout likewise (one
    // lane: 464 -> 435 us; B = 8 over two lanes: 934 -> 872 us, 923 with nw = 2);
    // bf16 8-byte rows lost 2-6 % (nw = 4 over two lanes: -1.3 %, not kept).
    // Forward: nw = 4 when a neuron spans several lanes (cifar 411 -> 395 us), 2
    // for fp32 with one lane per neuron and 16-byte rows (P = 4 on B = 2: 209 ->
    // 199 us; 4 no better), 1 for wider one-lane fp32 rows in the
    // compartments-innermost layout (twice the waves at three per SIMD; ten
    // compartments, T = 10: 175.8 -> 171.2 us Stateless, 206.8 -> 198.9 us
    // stateful; the channel-major cifar layer's one-lane forward keeps 2: 417
    // against 453 us); one-lane bf16 neurons and channel-major neurons over
    // several lanes gained nothing and keep 1.
    int nw = 1;
    if (bwd) {
      if (c->T == 4 && p.BL * p.KC * esz == 16) nw = L == 1 ? 2 : 4;
    } else if (L >= 2) {
      nw = p.cm ? 1 : 4;
    } else if (esz == 4) {
      nw = (!p.cm && p.BL * p.KC * esz > 16) ? 1 : 2;
    }
    while (nw > 1 && c->S % (nw * p.pb) != 0) nw /= 2;
    p.nw = nw;
    p.pb *= nw;
    p.tpc = int32_t(ceil_div(c->S, p.pb)); p.cpt = 1;
    p.ntiles = c->C * p.tpc;
  } else if (c->S == 1) {
    // Four batch ways of 64 / L channels, or in the backward of neurons over 8
    // or more lanes two ways of 128 / L channels: then each way's two waves read
    // adjacent halves of the same grad_spikes lines at about the same time (with
    // 8 channels a wave reads a quarter line per row).  Measured on MI355X: the
    // gated 32-branch layer's backward -3.6 % (twice the partial slots
    // included), the long-horizon layer (4 lanes) unchanged either way.
    p.mode = kFC; p.ways = (bwd && L >= 8) ? 2 : 4; p.pb = kThreads / (p.ways * L);
    p.tpc = 1; p.cpt = p.pb;
    p.ntiles = ceil_div(c->C, p.cpt);
  } else {
    p.mode = kSeg; p.ways = 1; p.pb = kThreads / L;
    p.tpc = 1; p.cpt = int32_t(p.pb / c->S);
    p.ntiles = ceil_div(c->C, p.cpt);
  }
  // Batch groups (measured on MI355X): the backward wants ~24K waves in the grid
  // for fp32 rows in the compartments-innermost layout (against ~16K: CIFAR-shaped
  // -0.5 to -1.1 %; ten compartments with 32K: +1-2 %), ~32K where such a row is
  // one lane's 16 bytes (P = 4 on B = 2 against ~24K: CIFAR-shaped -1.7 %, the
  // ResStateless layer -0.8 %; ~64K no better) and in the channel-major layout
  // (against ~16K: CIFAR-shaped -1.1 %, P = 4 on B = 2 -0.8 %; ~64K -0.4 % and
  // -2.8 %), and ~16K otherwise (with 24K: bf16 CIFAR +1.5 %); more groups mean
  // more partial sums to reduce.  The
  // forward over conv layers does best with one batch item per lane for fp32
  // (with the XCD eighths below: 1.5-4 % faster than two or four) and eight
  // neurons (batch items x positions) per lane for bf16 (4-5 % faster than four).
  const bool lane16 = esz == 4 && L == 1 && p.BL * p.KC * esz == 16;
  const int64_t target_waves = (p.cm || lane16) ? 32768 : (esz == 4 ? 24576 : 16384);
  int64_t G = ceil_div(target_waves, p.ntiles * 4);
  if (!bwd && p.mode == kSpatial) G = esz == 2 ? ceil_div(c->batch * p.nw, 8) : c->batch;
  // fully connected tiles (both directions): four batch items per wave (dbg: the
  // same as ~16K waves; long horizon, T = 64: forward -5 %, backward -3 %)
  if (p.mode == kFC) G = ceil_div(c->batch, int64_t(p.ways) * 4);
  G = G < 1 ? 1 : G;
  const int64_t max_g = ceil_div(c->batch, p.ways);
  if (G > max_g) G = max_g;
  if (bwd && p.mode != kSpatial && G > 8) G = 8;  // bounds the per-group partials
  if (c->batch_groups > 0) G = c->batch_groups < c->batch ? c->batch_groups : c->batch;
  p.bpg = int32_t(ceil_div(c->batch, G));
  p.G = int32_t(ceil_div(c->batch, p.bpg));
  const int64_t Ke = c->ckpt_every < c->T ? c->ckpt_every : c->T;
  p.nck = int32_t(ceil_div(c->T, c->ckpt_every) - 1);
  p.KS = (p.fast && p.KC == 1 && !p.cm && p.BL <= 4 && Ke >= 8) ? 8 : 4;
  // Occupancy cap (measured on MI355X): the backward over conv-shaped tiles whose
  // lanes move 16 bytes per row runs 3-4 % faster with at most two blocks per CU
  // (fewer concurrent streams contending for DRAM pages), and with two positions
  // per lane still 4 % faster when a neuron spans two or more lanes, but 1-2 %
  // slower with one lane per neuron; with 8-byte rows (bf16, four branches) or
  // the fully connected tiling the cap costs 15-17 %.  Unused dynamic LDS
  // reserves the room.
  // The stateful dendrite's wide fp32 lanes (more than 16 bytes of a row in a
  // lane) already hold about 70 KB of static LDS per block in the backward (the
  // DMA areas of their segment pipeline), which keeps them at two blocks per CU.
  const bool wide_sf = !p.cm && c->stateful && esz == 4 && p.BL * p.KC * esz > 16;
  const bool cap = bwd && p.mode == kSpatial && p.BL * p.KC * esz >= 16 && (p.nw == 1 || p.L >= 2) && !wide_sf;
  p.lds = cap ? int32_t(163840 / 3 + 256) : 0;
  // XCD runs (blocks are dealt to the 8 XCDs round-robin; measured on MI355X):
  // fully connected tiles in runs of 32 blocks per XCD (dbg forward / backward
  // -6 / -5 %, long horizon -5 / -3 %: neighbouring tiles share the cache lines
  // of their spike and grad_spikes rows), the fp32 forward over conv tiles one
  // contiguous eighth of the grid per XCD (cifar -4 %); otherwise round-robin
  // (with runs the conv backward and the bf16 stem lost 1-5 %).
  const int64_t nb = p.ntiles * p.G;
  int64_t xk = 1;
  if (p.mode == kFC) xk = 32;
  else if (!bwd && p.mode == kSpatial && esz == 4) xk = nb / 8;
  p.xk = (xk > 1 && nb % (8 * xk) == 0) ? int32_t(xk) : 1;
  return p;
}

// Checkpoints: the compartment states (stateful dendrite only) and the somatic
// potential after steps K, 2K, ... < T.
size_t ckpt_bytes(const dendsn_cfg* c, const Plan& p) {
  const int64_t N = c->batch * c->C * c->S;
  const size_t per_neuron = c->stateful ? size_t(c->B * c->comps_per_branch + 1) : 1;
  return size_t(p.nck) * size_t(N) * per_neuron * sizeof(float);
}

// Runtime kernel variant (see variant_bits).
int variant_of(const dendsn_cfg* c) { return c->psi | (c->residual << 1) | ((c->stateful ? 0 : 1) << 2); }

void ws_layout(const dendsn_cfg* c, const Plan& p, size_t* offA, size_t* total) {
  const size_t nP = size_t(p.G) * size_t(p.tpc) * size_t(c->C) * size_t(2 * c->B + c->B * c->comps_per_branch);
  const size_t nA = size_t(p.G) * size_t(p.ntiles);
  *offA = ((nP * sizeof(float) + 255) / 256) * 256;
  *total = *offA + 2 * nA * sizeof(float);  // g_alpha partials, then g_beta partials
}

dendsn_status check_grid(const dendsn_cfg* c, const Plan& p) {
  if (p.ntiles * p.G > int64_t(INT32_MAX)) return fail(DENDSN_E_UNSUPPORTED, "grid too large");
  const int64_t P = int64_t(c->B) * c->comps_per_branch;
  if (c->C * (2 * c->B + P) / (kThreads / 64) + 2 > int64_t(INT32_MAX))
    return fail(DENDSN_E_UNSUPPORTED, "too many parameter-gradient outputs");
  // per-lane byte offsets inside one sample's slice are 32-bit
  if (c->C * c->S * P * 4 > int64_t(UINT32_MAX)) return fail(DENDSN_E_UNSUPPORTED, "sample slice above 4 GiB");
  return DENDSN_OK;
}

void fill_scan(const dendsn_cfg* c, const Plan& p, const void* x, const float* alpha, const float* beta,
               const float* kappa, const float* xi, const float* zeta, const uint8_t* mask, ScanArgs* s) {
  s->x = x;
  s->alpha = c->stateful ? alpha : nullptr;
  s->beta_p = beta;
  s->rP = 1.0f / float(c->B * c->comps_per_branch);
  s->kappa = kappa; s->xi = xi; s->zeta = zeta; s->mask = mask;
  s->T = c->T; s->C = c->C; s->S = c->S; s->batch = c->batch;
  s->M = c->C * c->S; s->N = c->batch * s->M;
  s->B = c->B;
  s->P = c->B * c->comps_per_branch;
  s->xes = uint32_t((p.cm ? c->S : 1) * (c->io == DENDSN_IO_BF16 ? 2 : 4));
  s->K = int32_t(c->ckpt_every < c->T ? c->ckpt_every : c->T);
  s->nck = p.nck;
  s->beta = c->beta; s->vth = c->v_th;
  s->mode = p.mode; s->ways = p.ways; s->pb = p.pb; s->tpc = p.tpc; s->cpt = p.cpt; s->nw = p.nw;
  s->xk = p.xk;
  s->stg = !p.cm && (s->M * s->P * (c->io == DENDSN_IO_BF16 ? 2 : 4)) % 16 == 0;
  s->bpg = p.bpg; s->ntiles = p.ntiles;
}

}  // namespace

extern "C" {

const char* dendsn_status_str(dendsn_status st) {
  switch (st) {
    case DENDSN_OK: return "DENDSN_OK";
    case DENDSN_E_INVALID: return "DENDSN_E_INVALID";
    case DENDSN_E_UNSUPPORTED: return "DENDSN_E_UNSUPPORTED";
    case DENDSN_E_WORKSPACE: return "DENDSN_E_WORKSPACE";
    case DENDSN_E_HIP: return "DENDSN_E_HIP";
  }
  return "DENDSN_UNKNOWN_STATUS";
}

const char* dendsn_last_error(void) { return g_last_error.c_str(); }

dendsn_status dendsn_ckpt_bytes(const dendsn_cfg* cfg, size_t* bytes) {
  g_last_error.clear();
  dendsn_status st = check_cfg(cfg);
  if (st != DENDSN_OK) return st;
  if (!bytes) return fail(DENDSN_E_INVALID, "bytes is NULL");
  *bytes = empty_layer(cfg) ? 0 : ckpt_bytes(cfg, make_plan(cfg, false));
  return DENDSN_OK;
}

dendsn_status dendsn_bwd_workspace_bytes(const dendsn_cfg* cfg, size_t* bytes) {
  g_last_error.clear();
  dendsn_status st = check_cfg(cfg);
  if (st != DENDSN_OK) return st;
  if (!bytes) return fail(DENDSN_E_INVALID, "bytes is NULL");
  if (empty_layer(cfg)) {
    *bytes = kEmptyWorkspace;
    return DENDSN_OK;
  }
  size_t offA, total;
  ws_layout(cfg, make_plan(cfg, true), &offA, &total);
  *bytes = total;
  return DENDSN_OK;
}

dendsn_status dendsn_forward(const dendsn_cfg* cfg, const void* x, const float* alpha, const float* beta,
                             const float* kappa, const float* xi, const float* zeta, const uint8_t* mask,
                             void* spikes, float* v_soma, float* ckpt, hipStream_t stream) {
  g_last_error.clear();
  dendsn_status st = check_cfg(cfg);
  if (st != DENDSN_OK) return st;
  const bool empty = empty_layer(cfg);  // arrays of no elements may be NULL
  if (!x && !empty) return fail(DENDSN_E_INVALID, "x is NULL");
  if (!kappa && cfg->C > 0) return fail(DENDSN_E_INVALID, "kappa is NULL");
  if (!spikes && !empty) return fail(DENDSN_E_INVALID, "spikes is NULL");
  if (cfg->stateful && !alpha) return fail(DENDSN_E_INVALID, "alpha is NULL for a stateful dendrite");
  const size_t esz = cfg->io == DENDSN_IO_BF16 ? 2 : 4;
  if (!aligned(x, 16)) return fail(DENDSN_E_INVALID, "x must be 16-byte aligned");
  if (!aligned(spikes, esz)) return fail(DENDSN_E_INVALID, "spikes misaligned");
  if (ckpt && !aligned(ckpt, 16)) return fail(DENDSN_E_INVALID, "ckpt must be 16-byte aligned");
  if ((alpha && !aligned(alpha, 4)) || (beta && !aligned(beta, 4)) || !aligned(kappa, 4) ||
      (xi && !aligned(xi, 4)) || (zeta && !aligned(zeta, 4)) || (v_soma && !aligned(v_soma, 4)))
    return fail(DENDSN_E_INVALID, "fp32 tensor misaligned");
  if (empty) return DENDSN_OK;  // every output has no elements
  const Plan p = make_plan(cfg, false);
  if ((st = check_grid(cfg, p)) != DENDSN_OK) return st;
  FwdArgs fa;
  memset(&fa, 0, sizeof(fa));
  fill_scan(cfg, p, x, alpha, beta, kappa, xi, zeta, mask, &fa.s);
  fa.spikes = spikes;
  fa.vsoma = v_soma;
  float* ck = p.nck > 0 ? ckpt : nullptr;
  fa.ckpt = cfg->stateful ? ck : nullptr;
  fa.ckh = ck ? ck + (cfg->stateful ? int64_t(p.nck) * fa.s.N * fa.s.P : 0) : nullptr;
  const int v = variant_of(cfg);
  const bool bf = cfg->io == DENDSN_IO_BF16;
  const hipError_t e =
      p.cm ? (bf ? launch_fwd_bf16_cm(p, fa, v, stream) : launch_fwd_f32_cm(p, fa, v, stream))
      : p.KC == 1 ? (bf ? launch_fwd_bf16(p, fa, v, stream) : launch_fwd_f32(p, fa, v, stream))
                  : (bf ? launch_fwd_bf16_kc(p, fa, v, stream) : launch_fwd_f32_kc(p, fa, v, stream));
  if (e != hipSuccess) return fail(DENDSN_E_HIP, std::string("forward launch: ") + hipGetErrorString(e));
  return DENDSN_OK;
}

}  // extern "C"

namespace {

// ---------------------------------------------------------------------------
// The allocation-free backward's workspace: a device array of this module,
// one copy per GPU (each device that loads the library holds its own), whose
// address on the current device is looked up once per device.  Host code never
// passes `scratch` itself (in host code that name is a stand-in, not a device
// address); it passes the looked-up pointer.  The backward writes every partial
// slot it later reads within the call, so nothing needs clearing between calls.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = DENDSN_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

dendsn_status scratch_on_stream_device(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DENDSN_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return fail(DENDSN_E_HIP, std::string("hipStreamGetDevice: ") + hipGetErrorString(e));
    if (int(sdev) != dev)
      return fail(DENDSN_E_INVALID, "stream belongs to another device than the current one");
  }
  if (dev < 0 || dev >= kMaxDevices) return fail(DENDSN_E_UNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(DENDSN_E_HIP, std::string("scratch address: ") + hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DENDSN_OK;
}

// The backward of an empty layer: the finalize kernel over no partial slots
// writes +0 to every requested parameter gradient (a fill kernel, so the call
// records no memset node when captured into a graph).
dendsn_status zero_param_grads(const dendsn_cfg* cfg, const uint8_t* mask, float* grad_alpha, float* grad_beta,
                               float* grad_kappa, float* grad_xi, float* grad_zeta, hipStream_t stream) {
  FinArgs f;
  memset(&f, 0, sizeof(f));
  f.mask = mask;
  f.gk = grad_kappa; f.gxi = grad_xi; f.gz = grad_zeta; f.ga = grad_alpha; f.gb = grad_beta;
  f.C = cfg->C; f.B = cfg->B; f.P = cfg->B * cfg->comps_per_branch; f.KC = cfg->comps_per_branch;
  f.slots = 0; f.wide = 0; f.nA = 0;
  f.stateful = cfg->stateful;
  const int64_t nout = cfg->C * (2 * cfg->B + f.P);
  if (ceil_div(nout, kThreads) + 2 > int64_t(INT32_MAX))
    return fail(DENDSN_E_UNSUPPORTED, "too many parameter-gradient outputs");
  dendsn_finalize_kernel<<<dim3(unsigned(ceil_div(nout, kThreads) + 2)), dim3(kThreads), 0, stream>>>(f);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DENDSN_E_HIP, std::string("finalize launch: ") + hipGetErrorString(e));
  return DENDSN_OK;
}

// The backward on the caller's workspace or, with own_scratch, on the
// library's scratch array of the stream's device (every argument is checked
// before the array's address is looked up).
dendsn_status backward_impl(const dendsn_cfg* cfg, const void* x, const float* alpha, const float* beta,
                            const float* kappa, const float* xi, const float* zeta, const uint8_t* mask,
                            const float* ckpt, const void* grad_spikes, const float* grad_v_soma, void* grad_x,
                            float* grad_alpha, float* grad_beta, float* grad_kappa, float* grad_xi,
                            float* grad_zeta, void* workspace, size_t workspace_bytes, bool own_scratch,
                            hipStream_t stream) {
  dendsn_status st = check_cfg(cfg);
  if (st != DENDSN_OK) return st;
  const bool empty = empty_layer(cfg);  // arrays of no elements may be NULL
  if (!x && !empty) return fail(DENDSN_E_INVALID, "x is NULL");
  if (!kappa && cfg->C > 0) return fail(DENDSN_E_INVALID, "kappa is NULL");
  if (!grad_spikes && !empty) return fail(DENDSN_E_INVALID, "grad_spikes is NULL");
  if (!grad_x && !empty) return fail(DENDSN_E_INVALID, "grad_x is NULL");
  if (cfg->stateful && !alpha) return fail(DENDSN_E_INVALID, "alpha is NULL for a stateful dendrite");
  Plan p;
  memset(&p, 0, sizeof(p));
  if (!empty) p = make_plan(cfg, true);
  if (p.nck > 0 && !ckpt) return fail(DENDSN_E_INVALID, "ckpt is NULL but the forward wrote checkpoints");
  const size_t esz = cfg->io == DENDSN_IO_BF16 ? 2 : 4;
  if (!aligned(x, 16) || !aligned(grad_x, 16)) return fail(DENDSN_E_INVALID, "x / grad_x must be 16-byte aligned");
  if (ckpt && !aligned(ckpt, 16)) return fail(DENDSN_E_INVALID, "ckpt must be 16-byte aligned");
  if (!aligned(grad_spikes, esz)) return fail(DENDSN_E_INVALID, "grad_spikes misaligned");
  if ((alpha && !aligned(alpha, 4)) || (beta && !aligned(beta, 4)) || !aligned(kappa, 4) ||
      (xi && !aligned(xi, 4)) || (zeta && !aligned(zeta, 4)) || (grad_v_soma && !aligned(grad_v_soma, 4)) ||
      (grad_alpha && !aligned(grad_alpha, 4)) || (grad_beta && !aligned(grad_beta, 4)) ||
      (grad_kappa && !aligned(grad_kappa, 4)) ||
      (grad_xi && !aligned(grad_xi, 4)) || (grad_zeta && !aligned(grad_zeta, 4)))
    return fail(DENDSN_E_INVALID, "fp32 tensor misaligned");
  size_t offA = 0, total = kEmptyWorkspace;
  if (!empty) ws_layout(cfg, p, &offA, &total);
  if (own_scratch) {
    if (total > kScratchBytes)
      return fail(DENDSN_E_WORKSPACE, "layer needs " + std::to_string(total) +
                                          " workspace bytes, above the allocation-free scratch of " +
                                          std::to_string(kScratchBytes));
  } else {
    if (!workspace) return fail(DENDSN_E_WORKSPACE, "workspace is NULL");
    if (!aligned(workspace, 16)) return fail(DENDSN_E_WORKSPACE, "workspace must be 16-byte aligned");
    if (workspace_bytes < total)
      return fail(DENDSN_E_WORKSPACE, "workspace smaller than dendsn_bwd_workspace_bytes()");
  }
  if (empty) return zero_param_grads(cfg, mask, grad_alpha, grad_beta, grad_kappa, grad_xi, grad_zeta, stream);
  if ((st = check_grid(cfg, p)) != DENDSN_OK) return st;
  if (own_scratch && (st = scratch_on_stream_device(stream, &workspace)) != DENDSN_OK) return st;

  BwdArgs ba;
  memset(&ba, 0, sizeof(ba));
  fill_scan(cfg, p, x, alpha, beta, kappa, xi, zeta, mask, &ba.s);
  const float* ck = p.nck > 0 ? ckpt : nullptr;
  ba.ckpt = cfg->stateful ? ck : nullptr;
  ba.ckh = ck ? ck + (cfg->stateful ? int64_t(p.nck) * ba.s.N * ba.s.P : 0) : nullptr;
  ba.gspk = grad_spikes;
  ba.gv = grad_v_soma;
  // the single-chunk pipeline reads grad_v_soma through a buffer of gvn bytes:
  // with none, an empty buffer whose loads all return 0
  ba.gvz = grad_v_soma ? grad_v_soma : static_cast<const float*>(grad_spikes);
  ba.gvn = grad_v_soma ? 0xFFFFFFFFu : 0u;
  ba.gx = grad_x;
  ba.wsP = static_cast<float*>(workspace);
  ba.wsA = reinterpret_cast<float*>(static_cast<char*>(workspace) + offA);
  ba.wsB = ba.wsA + int64_t(p.G) * p.ntiles;
  ba.slots = int64_t(p.G) * p.tpc;
  ba.wide = ba.slots > kNarrowSlots;
  ba.detach = cfg->detach_reset;
  ba.sg_scale = cfg->sg_scale;
  const int v = variant_of(cfg);
  const bool bf = cfg->io == DENDSN_IO_BF16;
  hipError_t e;
  if (cfg->sg == DENDSN_SG_SIGMOID)
    e = p.cm ? (bf ? launch_bwd_bf16_cm_sg1(p, ba, v, stream) : launch_bwd_f32_cm_sg1(p, ba, v, stream))
        : p.KC == 1 ? (bf ? launch_bwd_bf16_sg1(p, ba, v, stream) : launch_bwd_f32_sg1(p, ba, v, stream))
                    : (bf ? launch_bwd_bf16_kc_sg1(p, ba, v, stream) : launch_bwd_f32_kc_sg1(p, ba, v, stream));
  else
    e = p.cm ? (bf ? launch_bwd_bf16_cm_sg0(p, ba, v, stream) : launch_bwd_f32_cm_sg0(p, ba, v, stream))
        : p.KC == 1 ? (bf ? launch_bwd_bf16_sg0(p, ba, v, stream) : launch_bwd_f32_sg0(p, ba, v, stream))
                    : (bf ? launch_bwd_bf16_kc_sg0(p, ba, v, stream) : launch_bwd_f32_kc_sg0(p, ba, v, stream));
  if (e != hipSuccess) return fail(DENDSN_E_HIP, std::string("backward launch: ") + hipGetErrorString(e));

  FinArgs f;
  memset(&f, 0, sizeof(f));
  f.wsP = ba.wsP; f.wsA = ba.wsA; f.wsB = ba.wsB; f.mask = mask;
  f.gk = grad_kappa; f.gxi = grad_xi; f.gz = grad_zeta; f.ga = grad_alpha; f.gb = grad_beta;
  f.C = cfg->C; f.B = cfg->B; f.P = ba.s.P; f.KC = p.KC; f.slots = ba.slots; f.wide = ba.wide;
  f.stateful = cfg->stateful;
  f.nA = int64_t(p.G) * p.ntiles;
  const int64_t nout = cfg->C * (2 * cfg->B + ba.s.P);
  const int64_t nblk = (f.wide ? ceil_div(nout, kThreads / 64) : ceil_div(nout, kThreads)) + 2;
  dendsn_finalize_kernel<<<dim3(unsigned(nblk)), dim3(kThreads), 0, stream>>>(f);
  e = hipGetLastError();
  if (e != hipSuccess) return fail(DENDSN_E_HIP, std::string("finalize launch: ") + hipGetErrorString(e));
  return DENDSN_OK;
}

}  // namespace

extern "C" {

dendsn_status dendsn_backward(const dendsn_cfg* cfg, const void* x, const float* alpha, const float* beta,
                              const float* kappa, const float* xi, const float* zeta, const uint8_t* mask,
                              const float* ckpt, const void* grad_spikes, const float* grad_v_soma,
                              void* grad_x, float* grad_alpha, float* grad_beta, float* grad_kappa,
                              float* grad_xi, float* grad_zeta, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  g_last_error.clear();
  return backward_impl(cfg, x, alpha, beta, kappa, xi, zeta, mask, ckpt, grad_spikes, grad_v_soma, grad_x,
                       grad_alpha, grad_beta, grad_kappa, grad_xi, grad_zeta, workspace, workspace_bytes, false,
                       stream);
}

dendsn_status dendsn_backward_noalloc(const dendsn_cfg* cfg, const void* x, const float* alpha,
                                      const float* beta, const float* kappa, const float* xi, const float* zeta,
                                      const uint8_t* mask, const float* ckpt, const void* grad_spikes,
                                      const float* grad_v_soma, void* grad_x, float* grad_alpha,
                                      float* grad_beta, float* grad_kappa, float* grad_xi, float* grad_zeta,
                                      hipStream_t stream) {
  g_last_error.clear();
  return backward_impl(cfg, x, alpha, beta, kappa, xi, zeta, mask, ckpt, grad_spikes, grad_v_soma, grad_x,
                       grad_alpha, grad_beta, grad_kappa, grad_xi, grad_zeta, nullptr, 0, true, stream);
}

}  // extern "C"
