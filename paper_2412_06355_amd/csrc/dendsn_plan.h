// Launch plan and kernel argument blocks shared by the host API and the kernel
// translation units.  Plain data only: no HIP runtime calls here.
#pragma once

#include <stdint.h>

namespace dendsn {

constexpr int kThreads = 256;  // 4 wave64s per block

// The backward translation units are compiled once per surrogate derivative
// (-DDENDSN_SG=0: atan, 1: sigmoid), which is bit 5 of the kernel variant V; their
// launchers carry the suffix _sg0 / _sg1.
#define DENDSN_SG_CAT2(name, k) name##_sg##k
#define DENDSN_SG_CAT(name, k) DENDSN_SG_CAT2(name, k)
#define DENDSN_SG_NAME(name) DENDSN_SG_CAT(name, DENDSN_SG)

// How the positions m = c * S + s of one sample are cut into per-block tiles.
// Tiles never straddle a channel unless they hold whole channels, so a block's
// parameter-gradient partials belong to a known set of channels.
enum TileMode : int32_t {
  kSpatial = 0,  // S >= positions per block: a tile is pb positions of ONE channel
  kFC = 1,       // S == 1: a tile is pb channels; the 4 waves split the batch items
  kSeg = 2,      // 1 < S < pb: a tile is cpt whole channels of S positions
};

struct Plan {
  int32_t BL;     // branches held by one lane
  int32_t L;      // lanes per neuron (power of two, <= 16); B = BL * L
  int32_t KC;     // compartments per branch (1, 2 or 4); a lane holds BL * KC of them
  int32_t cm;     // 1: channel-major X / grad_x (a neuron's compartments S apart)
  int32_t fast;   // 1: a vector-width mapping with every stash capacity compiled
  int32_t mode;   // TileMode
  int32_t ways;   // batch ways inside a block (waves that share positions)
  int32_t pb;     // positions per way in a block; pb * L * ways == kThreads
  int32_t tpc;    // tiles per channel (kSpatial), else 1
  int32_t cpt;    // channels per tile (kFC / kSeg), else 1
  int64_t ntiles; // tiles per sample
  int32_t G;      // batch groups (grid = ntiles * G blocks)
  int32_t bpg;    // batch items per group
  int32_t KS;     // backward stash capacity in steps (compile-time in the kernel)
  int32_t nck;    // interior checkpoints, ceil(T / K) - 1
  int32_t lds;    // dynamic LDS bytes per block, reserved only to cap blocks per CU
  int32_t nw;     // positions per lane and batch item in spatial tiles (1, 2 or 4)
  int32_t xk;     // XCD runs: consecutive tiles per XCD turn (1: plain round-robin)
};

struct ScanArgs {
  const void* x;
  const float* alpha;   // NULL for the Stateless Dendrite (alpha = 0)
  const float* kappa;
  const float* xi;      // NULL: 0
  const float* zeta;    // NULL: 1
  const uint8_t* mask;  // NULL: all branches kept
  const float* beta_p;  // learnable somatic decay on the device, or NULL: beta
  int64_t T, N, C, S, M, batch;  // M = C * S positions per sample
  int32_t B, P, K, nck;          // P = B * KC compartments per neuron
  uint32_t xes;                  // bytes between a neuron's compartments in X / grad_x
  float beta, vth;
  float rP;             // 1 / P (residual dendrite)
  int32_t mode, ways, pb, tpc, cpt, bpg;
  int32_t nw;           // spatial tiles: a lane takes positions p, p + 64 / L, ... (nw of them)
  int32_t xk;           // runs of xk consecutive blocks share an XCD (see locate)
  int32_t stg;          // 1: a sample's slice of X is a multiple of 16 bytes (wide rows may be staged)
  int64_t ntiles;
};

// Checkpoints (when nck > 0): [nck][N][P] dendritic states (the stateful
// dendrite only) followed by [nck][N] somatic potentials.
struct FwdArgs {
  ScanArgs s;
  void* spikes;
  float* vsoma;  // optional
  float* ckpt;   // [nck][N][P] dendritic states, or NULL (none kept, or the Stateless Dendrite)
  float* ckh;    // [nck][N] somatic potentials, or NULL (none kept)
};

struct BwdArgs {
  ScanArgs s;
  const float* ckpt;  // as FwdArgs
  const float* ckh;
  const void* gspk;
  const float* gv;  // optional
  void* gx;
  float* wsP;       // partial sums of (g_kappa, g_xi, g_zeta): `slots` per output, see partial_index
  float* wsA;       // [G][ntiles] partial sums of g_alpha
  float* wsB;       // [G][ntiles] partial sums of g_beta
  int64_t slots;    // partial slots per output: G * tpc
  int32_t wide;     // 1: output-major layout (slots > kNarrowSlots)
  int32_t detach;
  float sg_scale;
  const float* gvz;  // grad_v_soma, or any address when absent
  uint32_t gvn;      // bytes readable through gvz: 0xffffffff, or 0 when absent
};

struct FinArgs {
  const float* wsP;
  const float* wsA;
  const float* wsB;
  float* gb;
  const uint8_t* mask;
  float* gk;
  float* gxi;
  float* gz;
  float* ga;
  int64_t C, nA, slots;
  int32_t B, P, KC, wide, stateful;
};

constexpr int kNarrowSlots = 16;  // up to this many partial slots: one thread per output

// Runtime kernel variant v = psi | residual << 1 | stateless << 2, as the host
// passes it to the launchers, to the template variant bits (bits 0, 1, 6).
constexpr int variant_bits(int v) { return (v & 3) | ((v & 4) << 4); }
#define DENDSN_EACH_VARIANT(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7)

// Compiled (BL, L) mappings with one compartment per branch.  "Fast" mappings
// move 8 or 16 bytes per lane; "generic" ones cover other branch counts.  For
// powers of two the branch sum is the same balanced tree whatever the split
// of the neuron over lanes (pairwise in a lane, then the DPP butterfly), so
// the forward and the backward may split a neuron differently and still agree
// bit for bit.
// Backward stash capacities: 4 steps for every mapping, and 8 steps too when a
// lane holds at most 4 branches.
#define DENDSN_FAST_F32(X) X(4, 1) X(4, 2) X(4, 4) X(4, 8) X(4, 16)
// The fp32 forward also holds 8 branches per lane over two lanes (16 branches).
#define DENDSN_FAST_F32_FWD(X) DENDSN_FAST_F32(X) X(8, 2)
#define DENDSN_FAST_BF16(X) X(4, 1) X(8, 1) X(8, 2) X(8, 4) X(8, 8) X(8, 16)
// The bf16 backward also holds 4 branches per lane (8 bytes) up to 64 branches.
#define DENDSN_FAST_BF16_BWD(X) DENDSN_FAST_BF16(X) X(4, 2) X(4, 4) X(4, 8) X(4, 16)
#define DENDSN_GENERIC(X) X(1, 1) X(2, 1) X(3, 1) X(5, 1) X(6, 1) X(7, 1) X(5, 2) X(6, 2) X(7, 2)
#define DENDSN_GENERIC_KS 4

// Compiled (BL, L, KC) mappings with KC = 2 or 4 compartments per branch (stash
// capacity 4).  Fast ones put 16 bytes of compartments in a lane (BL KC = 4
// for fp32, 8 for bf16); generic ones hold a whole neuron of up to 14
// compartments in one lane.
#define DENDSN_KC_FAST_F32(X) X(2, 1, 2) X(2, 2, 2) X(2, 4, 2) X(2, 8, 2) X(2, 16, 2) \
                              X(1, 1, 4) X(1, 2, 4) X(1, 4, 4) X(1, 8, 4) X(1, 16, 4)
#define DENDSN_KC_FAST_BF16(X) X(4, 1, 2) X(4, 2, 2) X(4, 4, 2) X(4, 8, 2) X(4, 16, 2) \
                               X(2, 1, 4) X(2, 2, 4) X(2, 4, 4) X(2, 8, 4) X(2, 16, 4)
#define DENDSN_KC_GENERIC(X) X(1, 1, 2) X(2, 1, 2) X(3, 1, 2) X(5, 1, 2) X(6, 1, 2) X(7, 1, 2) \
                             X(1, 1, 4) X(2, 1, 4) X(3, 1, 4)

// Compiled (BL, L, KC) for the channel-major layout (stash capacity 4): the
// fewest lanes per neuron that leave at most 4 compartments in a lane with
// whole branches in each.
#define DENDSN_CM(X) X(1, 1, 1) X(2, 1, 1) X(3, 1, 1) X(4, 1, 1) X(5, 1, 1) X(7, 1, 1) X(3, 2, 1) \
                     X(4, 2, 1) X(4, 4, 1) X(1, 1, 2) X(2, 1, 2) X(3, 1, 2) X(2, 2, 2) X(2, 4, 2) \
                     X(1, 1, 4) X(1, 2, 4) X(1, 4, 4)
// The channel-major forward holds up to 8 compartments per lane: a power-of-two
// backward split with half the lanes (the same balanced branch-sum tree).
#define DENDSN_CM_FWD(X) DENDSN_CM(X) X(8, 1, 1) X(8, 2, 1) X(4, 1, 2) X(4, 2, 2) X(2, 1, 4) X(2, 2, 4)

}  // namespace dendsn
