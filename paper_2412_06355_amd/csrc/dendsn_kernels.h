// DendSN layer scan kernels for gfx950 (CDNA4, wave64).
//
// One kernel per direction.  A neuron's B branches (P = B KC compartments) are
// held by L adjacent lanes of one wavefront, BL = B / L whole branches per lane,
// so one time step of X for a wave is one contiguous, fully coalesced stretch of
// [T, N, P] memory (or, in the channel-major layout, KC BL accesses that are each
// contiguous across the wave).  The dendritic states stay in registers across
// the time loop; the only cross-lane traffic is the branch-to-soma sum Z,
// reduced with DPP inside the L-lane group, and every lane of the group then
// runs the soma redundantly (no broadcast).
//
// A block owns a tile of positions of one sample (see TileMode) and loops over a
// group of batch items, so per-channel parameters are loaded once per lane and
// parameter-gradient partials are summed in registers across those items.
//
// The forward kernel and the backward kernel's recompute of the forward call
// the same inline step functions, so (compiled with -ffp-contract=off, explicit
// fmaf and the raw v_exp_f32) they reproduce bit-identical states and spikes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dendsn_plan.h"

namespace dendsn {

typedef uint16_t bf16_t;  // bf16 storage

// Kernel variant V: bit 0 = Mexican-hat activation (else identity), bit 1 =
// residual dendrite (Z also receives the mean synaptic input of the neuron),
// bits 2-3 = log2 of the compartments per branch KC (1, 2 or 4), bit 4 =
// channel-major X / grad_x ([T, batch, C, P, S]: a neuron's compartments S
// elements apart), bit 6 = Stateless Dendrite (a compartment's state is its
// input of the step: no leak, no dendritic state across steps or checkpoints,
// no adjoint recurrence and no alpha gradient).  A lane holds BL branches,
// i.e. E = BL * KC compartments of its neuron.
template <int V> constexpr bool kMH = (V & 1) != 0;
template <int V> constexpr bool kRes = (V & 2) != 0;
template <int V> constexpr int kKC = 1 << ((V >> 2) & 3);
template <int V> constexpr bool kCM = (V & 16) != 0;
template <int V> constexpr int kSG = (V >> 5) & 1;  // backward only: dendsn_sg surrogate
template <int V> constexpr bool kSL = (V & 64) != 0;
// Forward over bf16 rows without the residual dendrite: the branch gate is applied
// while the raw rows are widened (the residual sums every compartment's input,
// gated or not).  Measured: forward 2-2.5 % faster; the backward kept its
// per-step select (there the change was neutral to 1.4 % slower).
template <typename IO, int V> constexpr bool kGateIn = sizeof(IO) == 2 && !kRes<V>;
// The branch sum takes a lane's branches in fused pairs (one multiply and one
// fused multiply-add per pair) when a lane holds at least two.  Every split of
// a neuron that the two directions and the two layouts use holds whole pairs in
// a lane whenever one of them does, except with four compartments per branch
// (the channel-major backward then holds one branch per lane, its forward two),
// which keeps the plain tree: the branch sum stays one tree over the fused
// leaves, and the directions and layouts agree bit for bit.
template <int V, int BL> constexpr bool kFuse = BL >= 2 && kKC<V> < 4;

// -(1/2) log2(e): exp(-u^2/2) = exp2(u^2 * kNegHalfLog2e)
constexpr float kNegHalfLog2e = -0.721347520444481703680f;
constexpr float kLog2e = 1.442695040888963407360f;
constexpr float kPi = 3.141592653589793238463f;

// ---------------------------------------------------------------------------
// Storage conversions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two floats -> two bf16 in one dword, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  f32x2_t f = {a, b};
  bf16x2_t h = __builtin_convertvector(f, bf16x2_t);
  return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ bf16_t to_bf16(float a) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(a));
}

// Streaming loads are non-temporal: X, grad_spikes and checkpoints are read
// once per pass, so they should not displace anything in the caches.  A lane
// row of more than 16 bytes takes several loads that each touch every cache
// line of the wave's stretch; those use the default policy, so that the later
// loads of a row find the lines the first brought in (non-temporal, a copy of
// 40-byte lane pieces ran at 1.9 TB/s against 4.6-4.9 with the default policy).
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// The policy is a template parameter: as a runtime flag, callers of one
// instance with both values let the compiler merge its two loads of the same
// address into one plain load, which dropped the non-temporal hint for every
// caller (the fp32 CIFAR forward, 16-byte rows, ran 14 % slower once a wide
// fp32 mapping shared its 16-byte load instance).
template <bool kCached, typename T>
__device__ __forceinline__ T stream_load(const T* p);

template <int BL>
__device__ __forceinline__ void load_vec(const float* __restrict__ p, float (&v)[BL]) {
  constexpr bool wide = BL * 4 > 16;
  if constexpr (BL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 4; ++i) {
      const f32x4_t q = stream_load<wide>(reinterpret_cast<const f32x4_t*>(p) + i);
      v[4 * i] = q.x; v[4 * i + 1] = q.y; v[4 * i + 2] = q.z; v[4 * i + 3] = q.w;
    }
  } else if constexpr (BL % 2 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 2; ++i) {
      const f32x2_t q = stream_load<wide>(reinterpret_cast<const f32x2_t*>(p) + i);
      v[2 * i] = q.x; v[2 * i + 1] = q.y;
    }
  } else {
#pragma unroll
    for (int i = 0; i < BL; ++i) v[i] = stream_load<wide>(p + i);
  }
}

template <int BL>
__device__ __forceinline__ void store_vec(float* __restrict__ p, const float (&v)[BL]) {
  if constexpr (BL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 4; ++i)
      reinterpret_cast<float4*>(p)[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
  } else if constexpr (BL % 2 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 2; ++i) reinterpret_cast<float2*>(p)[i] = make_float2(v[2 * i], v[2 * i + 1]);
  } else {
#pragma unroll
    for (int i = 0; i < BL; ++i) p[i] = v[i];
  }
}

// Address = wave-uniform base (scalar registers) + 32-bit per-lane byte offset.
template <typename P>
__device__ __forceinline__ P* at(P* base, uint32_t off) {
  return reinterpret_cast<P*>(reinterpret_cast<char*>(base) + off);
}
template <typename P>
__device__ __forceinline__ const P* at(const P* base, uint32_t off) {
  return reinterpret_cast<const P*>(reinterpret_cast<const char*>(base) + off);
}


// ---------------------------------------------------------------------------
// Streamed rows through buffer resources: the row base is wave-uniform (scalar
// registers, the resource), the lane's part a 32-bit offset, and a further
// uniform part rides in the instruction's scalar offset, so no per-lane 64-bit
// address arithmetic is spent on the backward's X, grad_spikes and grad_x rows.  Accesses
// are non-temporal (each byte is touched once per pass).
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kAuxNT = 2;  // cache policy: non-temporal (streaming)
// s_waitcnt vmcnt(0), other counters untouched: every vector memory access of
// the wave has completed.
constexpr int kWaitVmem = 0x0F70;


__device__ __forceinline__ rsrc_t make_rsrc(const void* base) {
  // raw buffer, byte range 4 GiB - 1 (every lane offset is a uint32 below it)
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, -1, 0x00020000);
}

// A raw buffer of `bytes` bytes: loads at or past the end return 0 without
// touching memory (bytes = 0 makes every load a zero).
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), 0x00020000);
}

// A wave-uniform value the compiler cannot prove uniform (a select on loop
// state inside the lanes' active region) made explicit: as part of a buffer
// resource it would otherwise be fed to the load through a per-lane loop over
// distinct values, whose first wait drains every request in flight.
__device__ __forceinline__ uint32_t uniform_u32(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

template <int BL>
__device__ __forceinline__ void bload_vec(rsrc_t r, uint32_t off, float (&v)[BL], const float*) {
  constexpr int kAuxNT = BL * 4 > 16 ? 0 : dendsn::kAuxNT;  // (see load_vec)
  if constexpr (BL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 4; ++i) {
      const u32x4_t q = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16u * i, 0, kAuxNT);
      v[4 * i] = __uint_as_float(q.x); v[4 * i + 1] = __uint_as_float(q.y);
      v[4 * i + 2] = __uint_as_float(q.z); v[4 * i + 3] = __uint_as_float(q.w);
    }
  } else if constexpr (BL % 2 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 2; ++i) {
      const u32x2_t q = __builtin_amdgcn_raw_buffer_load_b64(r, off + 8u * i, 0, kAuxNT);
      v[2 * i] = __uint_as_float(q.x); v[2 * i + 1] = __uint_as_float(q.y);
    }
  } else {
#pragma unroll
    for (int i = 0; i < BL; ++i) v[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off + 4u * i, 0, kAuxNT));
  }
}

template <int BL>
__device__ __forceinline__ void bload_vec(rsrc_t r, uint32_t off, float (&v)[BL], const bf16_t*) {
  constexpr int kAuxNT = BL * 2 > 16 ? 0 : dendsn::kAuxNT;  // (see load_vec)
  if constexpr (BL % 8 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 8; ++i) {
      const u32x4_t q = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16u * i, 0, kAuxNT);
      v[8 * i + 0] = bf16_lo(q.x); v[8 * i + 1] = bf16_hi(q.x);
      v[8 * i + 2] = bf16_lo(q.y); v[8 * i + 3] = bf16_hi(q.y);
      v[8 * i + 4] = bf16_lo(q.z); v[8 * i + 5] = bf16_hi(q.z);
      v[8 * i + 6] = bf16_lo(q.w); v[8 * i + 7] = bf16_hi(q.w);
    }
  } else if constexpr (BL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 4; ++i) {
      const u32x2_t q = __builtin_amdgcn_raw_buffer_load_b64(r, off + 8u * i, 0, kAuxNT);
      v[4 * i + 0] = bf16_lo(q.x); v[4 * i + 1] = bf16_hi(q.x);
      v[4 * i + 2] = bf16_lo(q.y); v[4 * i + 3] = bf16_hi(q.y);
    }
  } else if constexpr (BL % 2 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 2; ++i) {
      const uint32_t q = __builtin_amdgcn_raw_buffer_load_b32(r, off + 4u * i, 0, kAuxNT);
      v[2 * i] = bf16_lo(q); v[2 * i + 1] = bf16_hi(q);
    }
  } else {
#pragma unroll
    for (int i = 0; i < BL; ++i)
      v[i] = bf16_lo(uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, off + 2u * i, 0, kAuxNT)));
  }
}

template <int BL, int AUX = kAuxNT>
__device__ __forceinline__ void bstore_vec(rsrc_t r, uint32_t off, const float (&v)[BL], float*) {
  if constexpr (BL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 4; ++i) {
      const u32x4_t q = {__float_as_uint(v[4 * i]), __float_as_uint(v[4 * i + 1]), __float_as_uint(v[4 * i + 2]),
                         __float_as_uint(v[4 * i + 3])};
      __builtin_amdgcn_raw_buffer_store_b128(q, r, off + 16u * i, 0, AUX);
    }
  } else if constexpr (BL % 2 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 2; ++i) {
      const u32x2_t q = {__float_as_uint(v[2 * i]), __float_as_uint(v[2 * i + 1])};
      __builtin_amdgcn_raw_buffer_store_b64(q, r, off + 8u * i, 0, AUX);
    }
  } else {
#pragma unroll
    for (int i = 0; i < BL; ++i) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[i]), r, off + 4u * i, 0, AUX);
  }
}

template <int BL, int AUX = kAuxNT>
__device__ __forceinline__ void bstore_vec(rsrc_t r, uint32_t off, const float (&v)[BL], bf16_t*) {
  if constexpr (BL % 8 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 8; ++i) {
      const u32x4_t q = {pack_bf16x2(v[8 * i + 0], v[8 * i + 1]), pack_bf16x2(v[8 * i + 2], v[8 * i + 3]),
                         pack_bf16x2(v[8 * i + 4], v[8 * i + 5]), pack_bf16x2(v[8 * i + 6], v[8 * i + 7])};
      __builtin_amdgcn_raw_buffer_store_b128(q, r, off + 16u * i, 0, AUX);
    }
  } else if constexpr (BL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 4; ++i) {
      const u32x2_t q = {pack_bf16x2(v[4 * i + 0], v[4 * i + 1]), pack_bf16x2(v[4 * i + 2], v[4 * i + 3])};
      __builtin_amdgcn_raw_buffer_store_b64(q, r, off + 8u * i, 0, AUX);
    }
  } else if constexpr (BL % 2 == 0) {
#pragma unroll
    for (int i = 0; i < BL / 2; ++i)
      __builtin_amdgcn_raw_buffer_store_b32(pack_bf16x2(v[2 * i], v[2 * i + 1]), r, off + 4u * i, 0, AUX);
  } else {
#pragma unroll
    for (int i = 0; i < BL; ++i) __builtin_amdgcn_raw_buffer_store_b16(to_bf16(v[i]), r, off + 2u * i, 0, AUX);
  }
}

__device__ __forceinline__ float bload_one(rsrc_t r, uint32_t off, uint32_t soff, const float*) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, soff, kAuxNT));
}
__device__ __forceinline__ float bload_one(rsrc_t r, uint32_t off, uint32_t soff, const bf16_t*) {
  return bf16_lo(uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, off, soff, kAuxNT)));
}
__device__ __forceinline__ void bstore_one(rsrc_t r, uint32_t off, uint32_t soff, float v, float*) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, soff, kAuxNT);
}
__device__ __forceinline__ void bstore_one(rsrc_t r, uint32_t off, uint32_t soff, float v, bf16_t*) {
  __builtin_amdgcn_raw_buffer_store_b16(to_bf16(v), r, off, soff, kAuxNT);
}

// A lane's E compartments of X / grad_x in the row starting at `row`: adjacent
// (a vector access at the lane offset) or, in the channel-major layout, es
// bytes apart (one access each, the uniform i * es in the scalar offset; the
// lanes of a wave hold adjacent positions, so each access is contiguous across
// the wave).  Through a buffer resource: the backward's segment path.
template <int E, bool CM, typename IO>
__device__ __forceinline__ void load_x(const IO* row, uint32_t off, uint32_t es, float (&v)[E]) {
  const rsrc_t r = make_rsrc(row);
  if constexpr (CM) {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = bload_one(r, off, uint32_t(i) * es, row);
  } else {
    bload_vec<E>(r, off, v, row);
  }
}

template <int E, bool CM, typename IO>
__device__ __forceinline__ void store_gx(IO* row, uint32_t off, uint32_t es, const float (&v)[E]) {
  const rsrc_t r = make_rsrc(row);
  if constexpr (CM) {
#pragma unroll
    for (int i = 0; i < E; ++i) bstore_one(r, off, uint32_t(i) * es, v[i], row);
  } else {
    // Non-temporal up to 16 bytes a lane.  A longer row is several stores, each
    // writing every line it touches in pieces; as streaming stores the pieces
    // reached HBM separately (the ten-compartment fp32 rows wrote 32 % more
    // than grad_x, 1 % slower), so those go through L2 as default stores.
    // (Shorter multi-store rows, e.g. 12-byte bf16 ones, ran 1.7 % slower so.)
    constexpr bool streaming = E * sizeof(IO) <= 16;
    bstore_vec<E, streaming ? kAuxNT : 0>(r, off, v, row);
  }
}

// grad_x of one step, staged (see load_pieces): the lane's raw dwords go to the
// wave's LDS buffer and leave as whole 16-byte pieces, consecutive lanes on
// consecutive pieces (non-temporal: whole lines).
template <typename IO, int E>
__device__ __forceinline__ void store_gx_staged(IO* row, uint32_t span, const float (&v)[E], uint32_t* stage) {
  constexpr int W = sizeof(IO) == 4 ? E : E / 2;
  static_assert(sizeof(IO) == 4 || E % 2 == 0, "staged bf16 rows hold element pairs");
  const uint32_t lane = __lane_id();
#pragma unroll
  for (int j = 0; j < W; ++j)
    stage[lane * W + j] = sizeof(IO) == 4 ? __float_as_uint(v[j]) : pack_bf16x2(v[2 * j], v[2 * j + 1 < E ? 2 * j + 1 : 0]);
  __builtin_amdgcn_wave_barrier();
  const rsrc_t r = make_rsrc(row);
#pragma unroll
  for (int i = 0; i < (64 * W + 255) / 256; ++i) {
    const uint32_t d = (uint32_t(i) * 64 + lane) * 4;
    if (i < 64 * W / 256 || lane < (64 * W % 256) / 4)  // whole rounds, then the partial one
      __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4_t*>(stage + d), r, span + d * 4, 0, kAuxNT);
  }
  __builtin_amdgcn_wave_barrier();
}

template <typename IO>
__device__ __forceinline__ float load_row_one(const IO* row, uint32_t off) {
  return bload_one(make_rsrc(row), off, 0, row);
}

// ---------------------------------------------------------------------------
// Rows in raw form: the dwords the loads return (fp32 elements, bf16 element
// pairs, or one bf16 element in the low half), converted to float where they
// are used, so that the wait for a prefetched row falls at its first use and not
// right after its load.
// ---------------------------------------------------------------------------
template <typename IO, int E, bool CM>
constexpr int kRawW = (sizeof(IO) == 2 && !CM && E % 2 == 0) ? E / 2 : E;  // dwords per row

// Global (address) loads, as the forward issues them (non-temporal, except for
// lane rows of more than 16 bytes, as in bload_raw).
template <bool kCached, typename T>
__device__ __forceinline__ T stream_load(const T* p) {
  if constexpr (kCached) return *p;
  else return __builtin_nontemporal_load(p);
}

template <typename IO, int E, bool CM, int W>
__device__ __forceinline__ void load_raw(const IO* row, uint32_t off, uint32_t es, uint32_t (&w)[W]) {
  constexpr bool dwords = sizeof(IO) == 4 || (!CM && W * 2 == E);  // contiguous whole dwords
  constexpr bool wide = !CM && W * 4 > 16;
  if constexpr (CM) {
#pragma unroll
    for (int i = 0; i < W; ++i) {
      const IO* q = at(row, off + uint32_t(i) * es);
      if constexpr (sizeof(IO) == 4) w[i] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(q));
      else w[i] = uint32_t(__builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(q)));
    }
  } else if constexpr (dwords && W % 4 == 0) {
    const u32x4_t* q = reinterpret_cast<const u32x4_t*>(at(row, off));
#pragma unroll
    for (int i = 0; i < W / 4; ++i) {
      const u32x4_t v = stream_load<wide>(q + i);
      w[4 * i] = v.x; w[4 * i + 1] = v.y; w[4 * i + 2] = v.z; w[4 * i + 3] = v.w;
    }
  } else if constexpr (dwords && W % 2 == 0) {
    const u32x2_t* q = reinterpret_cast<const u32x2_t*>(at(row, off));
#pragma unroll
    for (int i = 0; i < W / 2; ++i) {
      const u32x2_t v = stream_load<wide>(q + i);
      w[2 * i] = v.x; w[2 * i + 1] = v.y;
    }
  } else if constexpr (dwords) {
    const uint32_t* q = reinterpret_cast<const uint32_t*>(at(row, off));
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = stream_load<wide>(q + i);
  } else {
    const uint16_t* q = reinterpret_cast<const uint16_t*>(at(row, off));
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = uint32_t(stream_load<wide>(q + i));
  }
}

// Buffer loads, as the backward issues them.  A lane row of more than 16 bytes
// takes several loads that each touch every cache line of the wave's row; those
// go through the caches with the default policy, so the later loads of a row
// find the lines the first one brought in.
template <typename IO, int E, bool CM, int W>
__device__ __forceinline__ void bload_raw(rsrc_t r, uint32_t off, uint32_t es, uint32_t (&w)[W]) {
  constexpr bool dwords = sizeof(IO) == 4 || (!CM && W * 2 == E);  // contiguous whole dwords
  constexpr int kAuxNT = (!CM && W * 4 > 16) ? 0 : dendsn::kAuxNT;
  if constexpr (CM) {
#pragma unroll
    for (int i = 0; i < W; ++i)
      w[i] = sizeof(IO) == 4 ? __builtin_amdgcn_raw_buffer_load_b32(r, off, uint32_t(i) * es, kAuxNT)
                             : uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, off, uint32_t(i) * es, kAuxNT));
  } else if constexpr (dwords && W % 4 == 0) {
#pragma unroll
    for (int i = 0; i < W / 4; ++i) {
      const u32x4_t q = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16u * i, 0, kAuxNT);
      w[4 * i] = q.x; w[4 * i + 1] = q.y; w[4 * i + 2] = q.z; w[4 * i + 3] = q.w;
    }
  } else if constexpr (dwords && W % 2 == 0) {
#pragma unroll
    for (int i = 0; i < W / 2; ++i) {
      const u32x2_t q = __builtin_amdgcn_raw_buffer_load_b64(r, off + 8u * i, 0, kAuxNT);
      w[2 * i] = q.x; w[2 * i + 1] = q.y;
    }
  } else if constexpr (dwords) {
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = __builtin_amdgcn_raw_buffer_load_b32(r, off + 4u * i, 0, kAuxNT);
  } else {
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, off + 2u * i, 0, kAuxNT));
  }
}

template <typename IO, int E, int W>
__device__ __forceinline__ void raw_to_float(const uint32_t (&w)[W], float (&v)[E]) {
  if constexpr (sizeof(IO) == 4) {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = __uint_as_float(w[i]);
  } else if constexpr (W * 2 == E) {
#pragma unroll
    for (int i = 0; i < W; ++i) { v[2 * i] = bf16_lo(w[i]); v[2 * i + 1] = bf16_hi(w[i]); }
  } else {
#pragma unroll
    for (int i = 0; i < E; ++i) v[i] = bf16_lo(w[i]);
  }
}

// v_perm_b32 byte selectors (result byte k <- selector byte k: 0-3 pick a byte
// of the dword, 0x0c gives 0x00): the bf16 in the low or high half widened to
// fp32 (low 16 bits zero), or +0.
constexpr uint32_t kPermLo = 0x01000C0Cu;
constexpr uint32_t kPermHi = 0x03020C0Cu;
constexpr uint32_t kPermZero = 0x0C0C0C0Cu;

// raw_to_float for bf16 rows with the branch gate folded in: one v_perm per
// element widens it, or zeroes it on a gated-off branch (so a gated branch's
// compartments integrate exact zeros and stay at +0 whatever the input holds).
template <int E, int W>
__device__ __forceinline__ void raw_to_float_gated(const uint32_t (&w)[W], const uint32_t (&sel)[E], float (&v)[E]) {
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const uint32_t d = w[W * 2 == E ? i / 2 : i];
    v[i] = __uint_as_float(__builtin_amdgcn_perm(d, d, sel[i]));
  }
}

template <typename IO>
__device__ __forceinline__ float raw_to_float(uint32_t w) {
  return sizeof(IO) == 4 ? __uint_as_float(w) : bf16_lo(w);
}

// ---------------------------------------------------------------------------
// Wide lane rows (more than 16 bytes of a row in one lane: the one-lane
// mappings of neurons with many compartments), staged.  Loaded lane by lane,
// each of a lane's several loads touches every cache line of the wave's
// stretch (a copy of 40-byte lane pieces ran 4.6-4.9 TB/s on MI355X against 5.7
// for 16-byte lanes, a read 5.9 against 6.3).  When the wave's 64 lanes hold one
// contiguous, 16-byte aligned stretch of 64 W dwords (every lane active), the
// wave moves the stretch as whole 16-byte pieces instead, consecutive lanes on
// consecutive pieces, and hands each lane its W dwords through a per-wave LDS
// buffer (ST = true below).
// ---------------------------------------------------------------------------
template <int W> constexpr int kPieces = (64 * W + 255) / 256;  // 16-byte pieces per lane
// Rows staged: a lane's row is more than 16 contiguous bytes that it keeps as
// whole dwords (fp32 elements or bf16 pairs; not the channel-major layout).
template <typename IO, int E, bool CM>
constexpr bool kWideRow = !CM && (sizeof(IO) == 4 || E % 2 == 0) && E * int(sizeof(IO)) > 16;
// dwords a lane keeps of one row: its W dwords, or its pieces when staged
template <int W, bool ST> constexpr int kSlotW = ST ? 4 * kPieces<W> : W;

// The pieces of the wave's stretch at byte `span` of `row` (non-temporal:
// whole lines); a piece past the stretch rereads the stretch's first.
// Round i of a stretch of 64 W dwords: lane l moves dwords 4 (64 i + l) ..
// + 3; every lane takes part in the first 64 W / 256 rounds, lanes below
// kTailLanes in the last, partial one.
template <int W> constexpr int kFullRounds = 64 * W / 256;
template <int W> constexpr uint32_t kTailLanes = (64 * W % 256) / 4;
template <int W>
__device__ __forceinline__ bool in_stretch(int i, uint32_t lane) {
  return i < kFullRounds<W> || lane < kTailLanes<W>;
}

template <typename IO, int W>
__device__ __forceinline__ void load_pieces(const IO* row, uint32_t span, uint32_t (&w)[4 * kPieces<W>]) {
  const uint32_t lane = __lane_id();
#pragma unroll
  for (int i = 0; i < kPieces<W>; ++i) {
    const uint32_t d = (uint32_t(i) * 64 + lane) * 4;
    const u32x4_t q = __builtin_nontemporal_load(
        reinterpret_cast<const u32x4_t*>(at(row, span + (in_stretch<W>(i, lane) ? d * 4 : 0u))));
    w[4 * i] = q.x; w[4 * i + 1] = q.y; w[4 * i + 2] = q.z; w[4 * i + 3] = q.w;
  }
}

// The same through a buffer resource (the backward's rows).
template <int W>
__device__ __forceinline__ void bload_pieces(rsrc_t r, uint32_t span, uint32_t (&w)[4 * kPieces<W>]) {
  const uint32_t lane = __lane_id();
#pragma unroll
  for (int i = 0; i < kPieces<W>; ++i) {
    const uint32_t d = (uint32_t(i) * 64 + lane) * 4;
    const u32x4_t q = __builtin_amdgcn_raw_buffer_load_b128(r, span + (in_stretch<W>(i, lane) ? d * 4 : 0u), 0, kAuxNT);
    w[4 * i] = q.x; w[4 * i + 1] = q.y; w[4 * i + 2] = q.z; w[4 * i + 3] = q.w;
  }
}

// The lane's W dwords out of the wave's pieces, through the wave's LDS buffer
// `stage` (64 W dwords).  LDS accesses of one wave complete in order.
template <int W>
__device__ __forceinline__ void pieces_to_lane(const uint32_t (&w)[4 * kPieces<W>], uint32_t* stage,
                                               uint32_t (&out)[W]) {
  const uint32_t lane = __lane_id();
#pragma unroll
  for (int i = 0; i < kPieces<W>; ++i) {
    const uint32_t d = (uint32_t(i) * 64 + lane) * 4;
    if (in_stretch<W>(i, lane)) *reinterpret_cast<u32x4_t*>(stage + d) = u32x4_t{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int j = 0; j < W; ++j) out[j] = stage[lane * W + j];
  __builtin_amdgcn_wave_barrier();
}

// A row slot (kSlotW dwords) as the lane's W raw dwords.
template <int W, bool ST>
__device__ __forceinline__ void slot_to_lane(const uint32_t (&slot)[kSlotW<W, ST>], uint32_t* stage, uint32_t (&out)[W]) {
  if constexpr (ST) {
    pieces_to_lane<W>(slot, stage, out);
  } else {
#pragma unroll
    for (int j = 0; j < W; ++j) out[j] = slot[j];
  }
}

// The same pieces moved by the memory unit straight into LDS (buffer loads
// with the LDS-DMA form): round i writes the 64 lanes' 16-byte pieces to dwords
// 256 i + 4 lane .. + 3 of `lds`, so the stretch's dword k lands at lds[k] and
// no register holds it in flight.  Lanes past the stretch in the last round
// request nothing, so a row's area is exactly its 64 W dwords.  The wave reads
// the area only after its vector memory counter has drained, and refills it
// only after its reads of it have completed (LDS reads and the DMA's LDS
// writes are not ordered otherwise).
template <int W> constexpr int kDmaDw = 64 * W;
typedef __attribute__((address_space(3))) void lds_void_t;
// s_waitcnt lgkmcnt(0), other counters untouched: every LDS access of the wave
// has completed.
constexpr int kWaitLds = 0xC07F;

// One round: the wave's 64 pieces at byte offsets `off` (per lane) into the 256
// dwords at `lds` (a plain function: the LDS-DMA builtin inside a template
// instantiated by the host compilation pass is rejected there).  Non-temporal,
// like every whole-line stream here (measured on MI355X, stateful P = 10
// backward: 375 -> 370 us alone, 388 -> 351 us back to back with the forward;
// with the default policy the X lines it leaves in the caches only served a
// forward of the same layer launched right after it, as no training step does).
__device__ __forceinline__ void dma_round(rsrc_t r, uint32_t off, uint32_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds, 16, off, 0, 0, kAuxNT);
}

template <int W>
__device__ __forceinline__ void dma_pieces(rsrc_t r, uint32_t span, uint32_t* lds) {
  const uint32_t lane = __lane_id();
#pragma unroll
  for (int i = 0; i < kPieces<W>; ++i) {
    const uint32_t d = (uint32_t(i) * 64 + lane) * 4;
    if (in_stretch<W>(i, lane)) dma_round(r, span + d * 4, lds + i * 256);
  }
}

__device__ __forceinline__ void store_spike(float* p, bool s) { *p = s ? 1.0f : 0.0f; }
__device__ __forceinline__ void store_spike(bf16_t* p, bool s) { *p = s ? bf16_t(0x3f80) : bf16_t(0); }

// ---------------------------------------------------------------------------
// Cross-lane sum inside an L-lane group (L <= 16) with DPP.  Every lane of the
// group ends with the same bits: each level adds a pair of partial sums that
// both partners hold, and float addition is commutative.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

template <int L>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(L == 1 || L == 2 || L == 4 || L == 8 || L == 16, "L must be a power of two <= 16");
  if constexpr (L >= 2) v += dpp_f32<0xb1>(v);   // quad_perm(1,0,3,2): partner lane ^ 1
  if constexpr (L >= 4) v += dpp_f32<0x4e>(v);   // quad_perm(2,3,0,1): partner lane ^ 2
  if constexpr (L >= 8) v += dpp_f32<0x141>(v);  // row_half_mirror: lane i <-> 7 - i in each 8
  if constexpr (L >= 16) v += dpp_f32<0x140>(v); // row_mirror: lane i <-> 15 - i in each 16
  return v;
}

// Pairwise tree over a lane's BL partial products (left fold for odd counts).
template <int BL>
__device__ __forceinline__ float lane_sum(const float (&p)[BL]) {
  if constexpr (BL == 1) {
    return p[0];
  } else if constexpr (BL == 2) {
    return p[0] + p[1];
  } else if constexpr (BL == 4) {
    return (p[0] + p[1]) + (p[2] + p[3]);
  } else if constexpr (BL == 8) {
    return ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
  } else {
    float s = p[0];
#pragma unroll
    for (int i = 1; i < BL; ++i) s += p[i];
    return s;
  }
}

// ---------------------------------------------------------------------------
// Per-lane branch parameters of one channel.
// ---------------------------------------------------------------------------
template <int BL, int KC>
struct Branches {
  float k[BL];        // kappa * m  (0 for a gated-off branch)
  float xi[BL * KC];  // per compartment
  float rz[BL];       // 1 / zeta
  float krz[BL];      // kappa* / zeta
  bool on[BL];        // mask bit
  float rp;           // 1 / P, the residual term's weight of each compartment
  // bf16 raw rows: v_perm selector per compartment that widens its bf16 half of
  // the dword to fp32, or yields 0 on a gated-off branch (see raw_to_float_gated)
  uint32_t xsel[BL * KC];
};

// packed_pairs: bf16 rows held as element pairs per dword (kRawW == E / 2)
template <int BL, int KC>
__device__ __forceinline__ void load_branches(const ScanArgs& a, int64_t c, int sub, Branches<BL, KC>& br,
                                              bool packed_pairs = false) {
  const int64_t base = c * a.B + int64_t(sub) * BL;
  const int64_t base_i = c * a.P + int64_t(sub) * (BL * KC);
  // Every load is issued before any value is used (the null checks are uniform
  // branches around whole groups), so the lot costs one memory round trip.
  float kap[BL], zet[BL];
  uint32_t msk[BL];
#pragma unroll
  for (int j = 0; j < BL; ++j) kap[j] = a.kappa[base + j];
  if (a.zeta) {
#pragma unroll
    for (int j = 0; j < BL; ++j) zet[j] = a.zeta[base + j];
  } else {
#pragma unroll
    for (int j = 0; j < BL; ++j) zet[j] = 1.0f;
  }
  if (a.mask) {
#pragma unroll
    for (int j = 0; j < BL; ++j) msk[j] = a.mask[base + j];
  } else {
#pragma unroll
    for (int j = 0; j < BL; ++j) msk[j] = 1;
  }
  if (a.xi) {
#pragma unroll
    for (int i = 0; i < BL * KC; ++i) br.xi[i] = a.xi[base_i + i];
  } else {
#pragma unroll
    for (int i = 0; i < BL * KC; ++i) br.xi[i] = 0.0f;
  }
#pragma unroll
  for (int j = 0; j < BL; ++j) {
    const bool on = msk[j] != 0;
    br.on[j] = on;
    br.k[j] = on ? kap[j] : 0.0f;
    br.rz[j] = 1.0f / zet[j];
    br.krz[j] = br.k[j] * br.rz[j];
  }
  br.rp = a.rP;
#pragma unroll
  for (int i = 0; i < BL * KC; ++i)
    br.xsel[i] = !br.on[i / KC] ? kPermZero : (packed_pairs && (i & 1) ? kPermHi : kPermLo);
}

// Sum of squares of a branch's KC compartment offsets d = Vd - xi, in a fixed order.
template <int KC>
__device__ __forceinline__ float branch_sumsq(const float* vd, const float* xi) {
  float d = vd[0] - xi[0];
  float ss = d * d;
#pragma unroll
  for (int i = 1; i < KC; ++i) {
    d = vd[i] - xi[i];
    ss = fmaf(d, d, ss);
  }
  return ss;
}

// ---------------------------------------------------------------------------
// One forward step of the dendrite (leaky compartments, L2 aggregation over
// each branch's compartments, activation, weighted branch sum) and of the LIF
// soma.  A gated-off branch keeps a zero state (its input zeroed, or its state
// reset every step), so nothing it receives can reach the soma or its gradients.
// ---------------------------------------------------------------------------
// kGated: no select needed, because xv is already 0 on gated-off branches
// (their state then stays +0 by itself) or because every branch of the lane is
// on.  tfac / yfac (one compartment per branch, Mexican hat) receive each
// branch's signed (Vd - xi) / zeta and psi as rounded here, for the adjoint.
template <int BL, int L, int V, bool kGated = false>
__device__ __forceinline__ float dendrite_step(float (&vd)[BL * kKC<V>], const float (&xv)[BL * kKC<V>],
                                               const Branches<BL, kKC<V>>& br, float alpha,
                                               float* efac = nullptr, float* tfac = nullptr,
                                               float* yfac = nullptr) {
  constexpr int KC = kKC<V>;
  float part[BL];
#pragma unroll
  for (int j = 0; j < BL; ++j) {
#pragma unroll
    for (int i = j * KC; i < (j + 1) * KC; ++i) {
      const float v = kSL<V> ? xv[i] : fmaf(alpha, vd[i], xv[i]);
      vd[i] = (kGated || br.on[j]) ? v : 0.0f;
    }
    // KC = 1: the signed (Vd - xi)/zeta, u = |tt|; else u = ||Vd - xi|| / zeta >= 0
    float tt;
    if constexpr (KC == 1)
      tt = (vd[j] - br.xi[j]) * br.rz[j];
    else
      tt = __builtin_amdgcn_sqrtf(branch_sumsq<KC>(&vd[j * KC], &br.xi[j * KC])) * br.rz[j];
    float y;
    if constexpr (kMH<V>) {
      const float q = tt * tt;
      const float e = __builtin_amdgcn_exp2f(q * kNegHalfLog2e);
      if (efac) efac[j] = e;
      y = fmaf(-q, e, e);  // (1 - q) e
      if (tfac) tfac[j] = tt;
      if (yfac) yfac[j] = y;
    } else {
      y = KC == 1 ? fabsf(tt) : tt;
    }
    // branch pairs (2i, 2i+1) of a lane enter the sum as one fused leaf
    // kappa*_{2i+1} Y_{2i+1} + kappa*_{2i} Y_{2i}; an odd branch count folds left
    float pj = (kFuse<V, BL> && (BL % 2 == 0 ? (j & 1) : j > 0)) ? fmaf(br.k[j], y, part[j > 0 ? j - 1 : 0]) : br.k[j] * y;
    if constexpr (kRes<V>) {
#pragma unroll
      for (int i = j * KC; i < (j + 1) * KC; ++i) pj = fmaf(xv[i], br.rp, pj);  // every compartment feeds the residual
    }
    part[j] = pj;
  }
  if constexpr (kFuse<V, BL>) {
    if constexpr (BL % 2 == 0) {
      float leaf[BL / 2];
#pragma unroll
      for (int i = 0; i < BL / 2; ++i) leaf[i] = part[2 * i + 1];
      return group_sum<L>(lane_sum<BL / 2>(leaf));
    } else {
      return group_sum<L>(part[BL - 1]);
    }
  }
  return group_sum<L>(lane_sum<BL>(part));
}

__device__ __forceinline__ void soma_step(float& h, bool& s, float z, float beta, float vth) {
  h = s ? z : fmaf(beta, h, z);   // beta (1 - S[t-1]) H[t-1] + Z[t]
  s = h >= vth;                   // Theta(H - v_th), Theta(0) = 1
}

// Surrogate derivative of Theta at x = H - v_th, with a x log2(e) (or pi x)
// formed in one fused multiply-add from H; kind is a compile-time constant of
// each backward kernel (dendsn_sg).
__device__ __forceinline__ float surrogate(float h, float vth, int kind, float a) {
  if (kind == 1) {  // a sigma(a x) (1 - sigma(a x)) = a e / (1 + e)^2, e = exp(-|a x|), x = h - v_th
    const float ac = a * kLog2e;
    const float t = fmaf(h, ac, -ac * vth);  // a x log2(e)
    const float e = __builtin_amdgcn_exp2f(-fabsf(t));
    const float d = 1.0f + e;
    return a * e * __builtin_amdgcn_rcpf(d * d);
  }
  const float px = fmaf(h, kPi, -kPi * vth);  // pi x: 1 / (1 + pi^2 x^2)
  return __builtin_amdgcn_rcpf(fmaf(px, px, 1.0f));
}

// ---------------------------------------------------------------------------
// Where a thread sits: lane-in-neuron, position, batch way, group, channel.
// ---------------------------------------------------------------------------
struct Pos {
  int sub, p, way, g;
  int64_t c, m, tile;
  bool active;
};

template <int L>
__device__ __forceinline__ Pos locate(const ScanArgs& a) {
  Pos r;
  const int tid = threadIdx.x;
  r.sub = tid % L;
  const int q = tid / L;
  // nw > 1 (spatial tiles): each wave covers nw * 64 / L adjacent
  // positions, a lane taking slot q of each 64 / L stretch, so each of the nw
  // accesses per row is contiguous across the wave.
  constexpr int kSlots = 64 / L;
  r.p = a.nw > 1 ? (q / kSlots) * (a.nw * kSlots) + q % kSlots : q % a.pb;
  // Batch ways are whole waves (kFC: pb * L is 64 or 128) or a single way, so the way
  // index is wave-uniform; readfirstlane lets the compiler keep it scalar.
  r.way = __builtin_amdgcn_readfirstlane(q / a.pb);
  // Blocks are dealt to the 8 XCDs round-robin; with xk > 1 block b takes the
  // tile of b's slot in runs of xk consecutive tiles per XCD turn, so tiles
  // that share cache lines (and neighbouring DRAM pages) meet in one XCD's L2.
  int64_t blk = blockIdx.x;
  if (a.xk > 1) {
    const int64_t x = blk % 8, j = blk / 8;
    blk = (j / a.xk) * (8 * int64_t(a.xk)) + x * a.xk + j % a.xk;
  }
  r.tile = blk % a.ntiles;
  r.g = int(blk / a.ntiles);
  if (a.mode == kSpatial) {
    const int64_t c = r.tile / a.tpc;
    const int64_t s = (r.tile % a.tpc) * a.pb + r.p;
    r.c = c;
    r.active = s < a.S;
    r.m = c * a.S + s;
  } else {
    const int64_t c = r.tile * a.cpt + r.p / a.S;
    r.c = c;
    r.active = (r.p < int64_t(a.cpt) * a.S) && (c < a.C);
    r.m = c * a.S + r.p % a.S;
  }
  return r;
}

// ---------------------------------------------------------------------------
// Per-lane byte offsets of one neuron inside a sample's slice of a time row;
// every other part of an address is wave-uniform (scalar registers).
// ---------------------------------------------------------------------------
struct LaneOff {
  uint32_t x;   // X / grad_x element (I/O dtype)
  uint32_t c;   // checkpointed dendritic state (fp32)
  uint32_t s;   // spikes / grad_spikes (I/O dtype)
  uint32_t v;   // fp32 per-neuron rows (v_soma, grad_v_soma, checkpointed H)
  uint32_t xw;  // staged wide rows (see load_pieces): the wave's stretch in X / grad_x
};

template <typename IO, int E, bool CM>
__device__ __forceinline__ LaneOff lane_offsets(const ScanArgs& a, const Pos& pos) {
  LaneOff o;
  // channel-major: compartment i of position s = m - c S of channel c sits at
  // (c P + i) S + s; this lane's first compartment is i = sub E
  o.x = CM ? uint32_t((pos.m + pos.c * (a.P - 1) * a.S + int64_t(pos.sub) * E * a.S) * int64_t(sizeof(IO)))
           : uint32_t((pos.m * a.P + pos.sub * E) * int64_t(sizeof(IO)));
  o.c = uint32_t((pos.m * a.P + pos.sub * E) * 4);
  o.s = uint32_t(pos.m * int64_t(sizeof(IO)));
  o.v = uint32_t(pos.m * 4);
  return o;
}

// Batch items of one lane: bt = first, first + ways, ... < end (wave-uniform).
__device__ __forceinline__ int items_of(const ScanArgs& a, const Pos& pos, int64_t* first) {
  *first = int64_t(pos.g) * a.bpg + pos.way;
  const int64_t end = min(a.batch, int64_t(pos.g + 1) * a.bpg);
  return *first < end ? int((end - *first + a.ways - 1) / a.ways) : 0;
}

// A lane's walk over its neurons when it holds nw > 1 positions per batch item
// (neurons n, n + 64 / L, ... of the item, then the next item): the wave-uniform
// shifts of the [T, N] row index n and of the matching X element offset nx (n P,
// or in the channel-major layout the item's base plus the position shift).
struct Walk {
  int nw;
  int64_t dn, dnx, dn_item, dnx_item;
};

template <int L, bool CM>
__device__ __forceinline__ Walk make_walk(const ScanArgs& a, int64_t item_neurons) {
  Walk k;
  k.nw = a.nw > 1 ? a.nw : 1;
  k.dn = 64 / L;
  k.dnx = CM ? k.dn : k.dn * a.P;
  k.dn_item = item_neurons - (k.nw - 1) * k.dn;
  k.dnx_item = item_neurons * a.P - (k.nw - 1) * k.dnx;
  return k;
}

// ---------------------------------------------------------------------------
// Forward kernel.
//
// Each lane walks the rows X[t] of its neurons (one neuron per batch item) as
// one stream, in chunks of D rows, double-buffered: chunk c+1 is in flight
// while chunk c is computed.  A neuron's rows are padded to a multiple of D by
// re-reading its last row; padded steps compute but store nothing, and the
// state restarts at each neuron's first chunk.
// ---------------------------------------------------------------------------
template <typename IO, int BL, int D>
struct RowCursor {  // wave-uniform position of the next chunk to load
  const IO* base;   // X row 0 of the current neuron's batch item
  int w, t;         // position index inside the item (0 .. nw-1), first row of the chunk
};

template <bool CM, bool ST, typename IO, int BL, int D>
__device__ __forceinline__ void load_chunk(const ScanArgs& a, RowCursor<IO, BL, D>& cur, uint32_t ox, int T,
                                           int Tp, int64_t rowX, const Walk& wk,
                                           uint32_t (&buf)[D][kSlotW<kRawW<IO, BL, CM>, ST>]) {
#pragma unroll
  for (int k = 0; k < D; ++k) {
    // A padding step past T (its result is discarded): every lane reads the
    // start of row T - 1, one cache line per wave instead of a whole row
    // (staged: the first stretch of the row).
    const int tk = cur.t + k;
    const int t = min(tk, T - 1);
    if constexpr (ST)
      load_pieces<IO, kRawW<IO, BL, CM>>(cur.base + int64_t(t) * rowX, tk < T ? ox : 0u, buf[k]);
    else
      load_raw<IO, BL, CM>(cur.base + int64_t(t) * rowX, tk < T ? ox : 0u, a.xes, buf[k]);
  }
  cur.t += D;
  if (cur.t >= Tp) {
    cur.t = 0;
    const bool last = ++cur.w == wk.nw;
    if (last) cur.w = 0;
    cur.base += last ? wk.dnx_item : wk.dnx;
  }
}

// Running state of the neuron a lane is computing, and wave-uniform output
// pointers of its batch item (advanced step by step, never recomputed).
template <typename IO, int E>
struct FwdLane {
  float vd[E];
  float h;
  bool s;
  int t;          // step index of the chunk being computed (0 .. Tp-1)
  int w;          // position index inside the batch item (0 .. nw-1)
  int kc;         // steps until the next checkpoint
  IO* sp;         // spikes row t of this batch item
  float* vp;      // v_soma row t (or null)
  float* ckv;     // next checkpoint's dendritic-state block of this item (stateful dendrite)
  float* ckh;     // next checkpoint's H row of this item
};

template <typename IO, int E>
__device__ __forceinline__ void fwd_item_start(const FwdArgs& fa, int64_t n0, FwdLane<IO, E>& st) {
  const ScanArgs& a = fa.s;
  st.t = 0;
  st.kc = a.K;
  st.sp = static_cast<IO*>(fa.spikes) + n0;
  st.vp = fa.vsoma ? fa.vsoma + n0 : nullptr;
  st.ckv = fa.ckpt ? fa.ckpt + n0 * a.P : nullptr;
  st.ckh = fa.ckh ? fa.ckh + n0 : nullptr;
#pragma unroll
  for (int j = 0; j < E; ++j) st.vd[j] = 0.0f;
  st.h = 0.0f;
  st.s = false;
}

template <typename IO, int BL, int L, int V, int D, bool ST>
__device__ __forceinline__ void compute_chunk(const FwdArgs& fa, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                              float alpha, bool lead, int T, int Tp, const Walk& wk,
                                              const uint32_t (&buf)[D][kSlotW<kRawW<IO, BL * kKC<V>, kCM<V>>, ST>],
                                              uint32_t* stage, FwdLane<IO, BL * kKC<V>>& st) {
  constexpr int E = BL * kKC<V>;
  constexpr int W = kRawW<IO, E, kCM<V>>;
  const ScanArgs& a = fa.s;
#pragma unroll
  for (int k = 0; k < D; ++k) {
    const int t = st.t + k;
    float xk[E];
    uint32_t raw[W];
    slot_to_lane<W, ST>(buf[k], stage, raw);
    if constexpr (kGateIn<IO, V>) raw_to_float_gated(raw, br.xsel, xk);
    else raw_to_float<IO, E>(raw, xk);
    const float z = dendrite_step<BL, L, V, kGateIn<IO, V>>(st.vd, xk, br, alpha);
    soma_step(st.h, st.s, z, a.beta, a.vth);
    if (t < T) {  // padded steps store nothing
      if (lead) {
        store_spike(at(st.sp, lo.s), st.s);
        if (st.vp) *at(st.vp, lo.v) = st.h;
      }
      if (--st.kc == 0) {
        st.kc = a.K;
        if (st.ckh && t + 1 < T) {
          if constexpr (!kSL<V>) {  // the Stateless Dendrite has no state to keep
            store_vec<E>(at(st.ckv, lo.c), st.vd);
            st.ckv += a.N * a.P;
          }
          if (lead) *at(st.ckh, lo.v) = st.h;
          st.ckh += a.N;
        }
      }
      st.sp += a.N;
      if (st.vp) st.vp += a.N;
    }
  }
  st.t += D;
  if (st.t >= Tp) {  // next neuron of this lane: next position of the item, or the next item
    const bool last = ++st.w == wk.nw;
    if (last) st.w = 0;
    const int64_t n0 = (st.sp - static_cast<IO*>(fa.spikes)) - int64_t(T) * a.N + (last ? wk.dn_item : wk.dn);
    fwd_item_start<IO, E>(fa, n0, st);
  }
}

// ---------------------------------------------------------------------------
// Forward fast path: T a multiple of D (no padding steps), no v_soma output and
// checkpoints, if any, only at chunk ends (K a multiple of D; the kernel takes
// it without interior checkpoints).  A step's bookkeeping is then the spike
// store alone: a row's address is the previous row's plus one row stride, and
// the checkpoint and next-neuron decisions are taken once per chunk.  A SIMD issues at most one scalar instruction per
// vector instruction slot, so the general path's per-step address arithmetic
// and conditions (more scalar than vector instructions per step) held the
// kernel back.
// ---------------------------------------------------------------------------
template <typename IO, int BL, int L, int V, int D, bool ST>
__device__ __forceinline__ void fwd_fast(const FwdArgs& fa, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                         float alpha, bool lead, int64_t bt0, int nk, const Walk& wk,
                                         uint32_t* stage) {
  constexpr int E = BL * kKC<V>;
  constexpr int W = kRawW<IO, E, kCM<V>>;
  constexpr int SW = kSlotW<W, ST>;
  const ScanArgs& a = fa.s;
  const int T = int(a.T), K = a.K;
  const int64_t rowX = a.N * a.P;
  const int nchunks = nk * wk.nw * (T / D);
  if (nchunks <= 0) return;
  // load cursor (wave-uniform): the next chunk's first row, the row 0 of that
  // chunk's neuron, its step and position index
  const IO* lrow = static_cast<const IO*>(a.x) + bt0 * a.M * a.P;
  const IO* lbase = lrow;
  int lt = 0, lw = 0;
  auto load = [&](uint32_t (&buf)[D][SW]) {
    const IO* r = lrow;
#pragma unroll
    for (int k = 0; k < D; ++k) {
      if constexpr (ST) load_pieces<IO, W>(r, lo.x, buf[k]);
      else load_raw<IO, E, kCM<V>>(r, lo.x, a.xes, buf[k]);
      r += rowX;
    }
    lt += D;
    if (lt == T) {
      lt = 0;
      const bool last = ++lw == wk.nw;
      if (last) lw = 0;
      lbase += last ? wk.dnx_item : wk.dnx;
      r = lbase;
    }
    lrow = r;
  };
  // the neuron being computed: state, step, position, output rows (uniform)
  IO* const spk = static_cast<IO*>(fa.spikes);
  int64_t n0 = bt0 * a.M;
  IO* sp = spk + n0;
  float* ckv = fa.ckpt ? fa.ckpt + n0 * a.P : nullptr;
  float* ckh = fa.ckh ? fa.ckh + n0 : nullptr;
  float vd[E];
#pragma unroll
  for (int j = 0; j < E; ++j) vd[j] = 0.0f;
  float h = 0.0f;
  bool s = false;
  int ct = 0, cw = 0, kc = K;
  auto compute = [&](const uint32_t (&buf)[D][SW]) {
#pragma unroll
    for (int k = 0; k < D; ++k) {
      float xk[E];
      uint32_t raw[W];
      slot_to_lane<W, ST>(buf[k], stage, raw);
      if constexpr (kGateIn<IO, V>) raw_to_float_gated(raw, br.xsel, xk);
      else raw_to_float<IO, E>(raw, xk);
      const float z = dendrite_step<BL, L, V, kGateIn<IO, V>>(vd, xk, br, alpha);
      soma_step(h, s, z, a.beta, a.vth);
      if (lead) store_spike(at(sp, lo.s), s);
      sp += a.N;
    }
    ct += D;
    kc -= D;
    if (kc == 0) {  // a checkpoint after this chunk's last step (none after the last step)
      kc = K;
      if (ckh && ct < T) {
        if constexpr (!kSL<V>) {
          store_vec<E>(at(ckv, lo.c), vd);
          ckv += a.N * a.P;
        }
        if (lead) *at(ckh, lo.v) = h;
        ckh += a.N;
      }
    }
    if (ct == T) {  // next neuron of this lane: next position of the item, or the next item
      ct = 0;
      kc = K;
      const bool last = ++cw == wk.nw;
      if (last) cw = 0;
      n0 += last ? wk.dn_item : wk.dn;
      sp = spk + n0;
      ckv = fa.ckpt ? fa.ckpt + n0 * a.P : nullptr;
      ckh = fa.ckh ? fa.ckh + n0 : nullptr;
#pragma unroll
      for (int j = 0; j < E; ++j) vd[j] = 0.0f;
      h = 0.0f;
      s = false;
    }
  };
  uint32_t bufA[D][SW], bufB[D][SW];
  load(bufA);
  // Every later wait is then counted from loads issued inside the loop, which
  // are unconditional (the last one or two chunks run after it).
  __builtin_amdgcn_s_waitcnt(kWaitVmem);
  int c = 0;
  for (; c + 2 < nchunks; c += 2) {
    load(bufB);
    compute(bufA);
    load(bufA);
    compute(bufB);
  }
  if (c + 1 < nchunks) {
    load(bufB);
    compute(bufA);
    compute(bufB);
  } else {
    compute(bufA);
  }
}

// The forward of the lane's neurons (ST: wide rows staged, see load_pieces;
// lo.x is then the wave's stretch, the same for every lane).
template <typename IO, int BL, int L, int V, int D, bool ST>
__device__ __forceinline__ void fwd_run(const FwdArgs& fa, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                        float alpha, bool lead, int64_t bt0, int nk, uint32_t* stage) {
  constexpr int E = BL * kKC<V>;
  constexpr int SW = kSlotW<kRawW<IO, E, kCM<V>>, ST>;
  const ScanArgs& a = fa.s;
  const int T = int(a.T);
  const int Tp = (T + D - 1) / D * D;
  const int64_t rowX = a.N * a.P;
  const Walk wk = make_walk<L, kCM<V>>(a, int64_t(a.ways) * a.M);
  // (with interior checkpoints, e.g. the T = 64 layer with K = 8, the general
  // path measured 2 % faster: those long sequences are bound by memory latency)
  if (T % D == 0 && !fa.vsoma && a.nck == 0) {
    fwd_fast<IO, BL, L, V, D, ST>(fa, lo, br, alpha, lead, bt0, nk, wk, stage);
    return;
  }
  const int nchunks = nk * wk.nw * (Tp / D);

  RowCursor<IO, E, D> cur;
  cur.base = static_cast<const IO*>(a.x) + bt0 * a.M * a.P;
  cur.w = 0;
  cur.t = 0;
  FwdLane<IO, E> st;
  st.w = 0;
  fwd_item_start<IO, E>(fa, bt0 * a.M, st);

  if (nchunks <= 0) return;
  uint32_t bufA[D][SW], bufB[D][SW];
  load_chunk<kCM<V>, ST>(a, cur, lo.x, T, Tp, rowX, wk, bufA);
  // Every later wait is then counted from loads issued inside the loop, which
  // are unconditional (the last one or two chunks run after it).
  __builtin_amdgcn_s_waitcnt(kWaitVmem);
  int c = 0;
  for (; c + 2 < nchunks; c += 2) {
    load_chunk<kCM<V>, ST>(a, cur, lo.x, T, Tp, rowX, wk, bufB);
    compute_chunk<IO, BL, L, V, D, ST>(fa, lo, br, alpha, lead, T, Tp, wk, bufA, stage, st);
    load_chunk<kCM<V>, ST>(a, cur, lo.x, T, Tp, rowX, wk, bufA);
    compute_chunk<IO, BL, L, V, D, ST>(fa, lo, br, alpha, lead, T, Tp, wk, bufB, stage, st);
  }
  if (c + 1 < nchunks) {
    load_chunk<kCM<V>, ST>(a, cur, lo.x, T, Tp, rowX, wk, bufB);
    compute_chunk<IO, BL, L, V, D, ST>(fa, lo, br, alpha, lead, T, Tp, wk, bufA, stage, st);
    compute_chunk<IO, BL, L, V, D, ST>(fa, lo, br, alpha, lead, T, Tp, wk, bufB, stage, st);
  } else {
    compute_chunk<IO, BL, L, V, D, ST>(fa, lo, br, alpha, lead, T, Tp, wk, bufA, stage, st);
  }
}

// Whether a wave may stage its wide rows: every lane active (checked by the
// caller), the layer's per-sample slice a multiple of 16 bytes (the host's
// flag: then every row and item keeps the alignment of the first), and the
// wave's first stretch 16-byte aligned.  lo.x of lane 0 is the stretch's start.
template <typename IO>
__device__ __forceinline__ bool stage_rows(const ScanArgs& a, uint32_t span0, int64_t bt0) {
  const uintptr_t p = reinterpret_cast<uintptr_t>(static_cast<const IO*>(a.x) + bt0 * a.M * a.P) + span0;
  return a.stg && (p & 15) == 0;
}

template <typename IO, int BL, int L, int V>
__global__ void __launch_bounds__(kThreads) dendsn_fwd_kernel(FwdArgs fa) {
  constexpr int D = 4;  // rows per chunk; two chunks in flight per lane
  if (fa.s.beta_p) fa.s.beta = fa.s.beta_p[0];  // learnable (PLIF) decay
  const ScanArgs& a = fa.s;
  const Pos pos = locate<L>(a);
  constexpr int E = BL * kKC<V>;
  constexpr int W = kRawW<IO, E, kCM<V>>;
  constexpr bool kWide = kWideRow<IO, E, kCM<V>>;
  const bool full = kWide && __all(pos.active);
  if (!pos.active) return;  // whole L-lane groups leave together
  Branches<BL, kKC<V>> br;
  load_branches<BL, kKC<V>>(a, pos.c, pos.sub, br, W * 2 == E);
  const float alpha = a.alpha ? a.alpha[0] : 0.0f;
  LaneOff lo = lane_offsets<IO, E, kCM<V>>(a, pos);
  const bool lead = pos.sub == 0;
  int64_t bt0;
  const int nk = items_of(a, pos, &bt0);
  if constexpr (kWide) {
    __shared__ uint32_t stage[kThreads / 64][64 * W];
    const uint32_t span = __builtin_amdgcn_readfirstlane(lo.x);
    if (full && stage_rows<IO>(a, span, bt0)) {
      lo.x = span;
      fwd_run<IO, BL, L, V, D, true>(fa, lo, br, alpha, lead, bt0, nk, stage[threadIdx.x >> 6]);
      return;
    }
  }
  fwd_run<IO, BL, L, V, D, false>(fa, lo, br, alpha, lead, bt0, nk, nullptr);
}

// ---------------------------------------------------------------------------
// Backward kernel.  For each neuron, the segments between checkpoints are
// visited from last to first.  A segment is cut into whole chunks of
// compile-time length (KS, then powers of two for the remainder); a chunk
// re-runs the forward from the segment's checkpoint up to its first step (only
// chunks after the first need that), recomputes its own steps while stashing
// the dendritic state and H in registers, then runs the adjoint recurrences
// backwards through them.
// ---------------------------------------------------------------------------
template <int BL, int E>
struct Accum {
  float k[BL], xi[E], z[BL];
  float a;   // g_alpha terms of this lane's branches
  float b;   // g_beta terms of this lane's neuron (counted by its first lane only)
};

template <typename IO, int E>
struct BwdLane {  // adjoint state carried backwards through time, and pointers
  float dh_next;
  float lam[E];
  uint32_t* stage;   // the wave's LDS buffer for staged wide rows (see load_pieces)
  const IO* xbase;   // X of this batch item (uniform)
  IO* gxbase;
  const IO* gsbase;
  const float* gvbase;
};

// The streamed inputs of one chunk of CS steps.
template <int E, int CS>
struct ChunkIn {
  float x[CS][E];
  float gs[CS];
  float gv[CS];
};

// grad_v_soma rows of a chunk (0 without grad_v_soma); issued with the chunk's
// other loads so no step waits on a load issued after its stores.
template <int E, int CS>
__device__ __forceinline__ void load_chunk_gv(const ScanArgs& a, const LaneOff& lo, const float* gvbase, int c0,
                                              ChunkIn<E, CS>& in) {
  if (gvbase) {
#pragma unroll
    for (int k = 0; k < CS; ++k) in.gv[k] = __builtin_nontemporal_load(at(gvbase + int64_t(c0 + k) * a.N, lo.v));
  } else {
#pragma unroll
    for (int k = 0; k < CS; ++k) in.gv[k] = 0.0f;
  }
}

template <typename IO, int E, int CS, bool CM>
__device__ __forceinline__ void load_chunk_in(const ScanArgs& a, const LaneOff& lo, const IO* xbase,
                                              const IO* gsbase, const float* gvbase, int c0, ChunkIn<E, CS>& in) {
  const int64_t rowX = a.N * a.P;
#pragma unroll
  for (int k = 0; k < CS; ++k) {
    const int64_t t = c0 + k;
    load_x<E, CM>(xbase + t * rowX, lo.x, a.xes, in.x[k]);
    in.gs[k] = load_row_one(gsbase + t * a.N, lo.s);
  }
  load_chunk_gv<E, CS>(a, lo, gvbase, c0, in);
}

// A chunk's rows in raw form (see load_raw).  The single-chunk pipeline
// carries the next neuron's rows this way: a conversion issued next to the
// loads would make the wave wait for them at once instead of while the current
// neuron's adjoint pass runs.
template <typename IO, int E, int CS, bool CM, bool ST = false>
struct ChunkRaw {
  uint32_t x[CS][kSlotW<kRawW<IO, E, CM>, ST>];
  uint32_t gs[CS];
  float gv[CS];
};

template <typename IO, int E, int CS, bool CM, bool GV = true, bool ST = false>
__device__ __forceinline__ void load_chunk_raw(const ScanArgs& a, const LaneOff& lo, const IO* xbase,
                                               const IO* gsbase, const float* gvbase, uint32_t gvbytes,
                                               ChunkRaw<IO, E, CS, CM, ST>& in) {
  const int64_t rowX = a.N * a.P;
#pragma unroll
  for (int k = 0; k < CS; ++k) {
    if constexpr (ST) bload_pieces<kRawW<IO, E, CM>>(make_rsrc(xbase + k * rowX), lo.xw, in.x[k]);
    else bload_raw<IO, E, CM>(make_rsrc(xbase + k * rowX), lo.x, a.xes, in.x[k]);
    const rsrc_t rg = make_rsrc(gsbase + k * a.N);
    in.gs[k] = sizeof(IO) == 4 ? __builtin_amdgcn_raw_buffer_load_b32(rg, lo.s, 0, kAuxNT)
                               : uint32_t(__builtin_amdgcn_raw_buffer_load_b16(rg, lo.s, 0, kAuxNT));
  }
  // grad_v_soma rows (a buffer of no bytes when absent: every load returns 0);
  // GV = false: known absent, nothing is requested
#pragma unroll
  for (int k = 0; k < CS; ++k)
    in.gv[k] = GV ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(make_rsrc(gvbase + int64_t(k) * a.N, gvbytes),
                                                                       lo.v, 0, kAuxNT))
                  : 0.0f;
}

// The checkpointed state a segment starts from.
template <int E>
struct SegStart {
  float v[E];
  float h;
};

template <typename IO, int E, bool SL>
__device__ __forceinline__ void load_seg_start(const BwdArgs& ba, const LaneOff& lo, int64_t n0, int seg,
                                               SegStart<E>& st) {
  const ScanArgs& a = ba.s;
  if (seg == 0 || SL) {  // the Stateless Dendrite restarts from its input: no state to load
#pragma unroll
    for (int j = 0; j < E; ++j) st.v[j] = 0.0f;
  } else {
    load_vec<E>(at(ba.ckpt + (int64_t(seg - 1) * a.N + n0) * a.P, lo.c), st.v);
  }
  st.h = seg == 0 ? 0.0f : __builtin_nontemporal_load(at(ba.ckh + int64_t(seg - 1) * a.N + n0, lo.v));
}

// Registers a chunk's recompute leaves for its adjoint pass: the dendritic
// state before and at each step, H at each step and, for the Mexican hat, the
// exp(-u^2/2) factor of each step.
template <int BL, int CS, int V>
struct Stash {
  float v[CS + 1][BL * kKC<V>];
  float e[kMH<V> ? CS : 1][BL];
  // one compartment per branch with the Mexican hat: the signed (Vd - xi) / zeta
  // and psi of each step, as the recompute rounded them
  float t[kMH<V> && kKC<V> == 1 ? CS : 1][BL];
  float y[kMH<V> && kKC<V> == 1 ? CS : 1][BL];
  float h[CS];
  float hd0;  // (1 - S) H before the chunk's first step: the decayed term beta multiplies
};

// Re-runs the chunk's forward steps exactly as the forward kernel did (the same
// inline step function, so the same bits).  NG: every branch of the lane is on
// (no gate select; with every branch on the select is the identity).
template <int BL, int L, int V, int CS, bool NG = false>
__device__ __forceinline__ void recompute_chunk(const ScanArgs& a, const Branches<BL, kKC<V>>& br, float alpha,
                                                const float (&v0)[BL * kKC<V>], float h0, bool s0,
                                                const float (&x)[CS][BL * kKC<V>], Stash<BL, CS, V>& st) {
  constexpr int E = BL * kKC<V>;
#pragma unroll
  for (int j = 0; j < E; ++j) st.v[0][j] = v0[j];
  st.hd0 = s0 ? 0.0f : h0;
  float h = h0;
  bool s = s0;
#pragma unroll
  for (int k = 0; k < CS; ++k) {
#pragma unroll
    for (int j = 0; j < E; ++j) st.v[k + 1][j] = st.v[k][j];
    constexpr bool ty = kMH<V> && kKC<V> == 1;
    const float z = dendrite_step<BL, L, V, NG>(st.v[k + 1], x[k], br, alpha, kMH<V> ? st.e[kMH<V> ? k : 0] : nullptr,
                                            ty ? st.t[ty ? k : 0] : nullptr, ty ? st.y[ty ? k : 0] : nullptr);
    soma_step(h, s, z, a.beta, a.vth);
    st.h[k] = h;
  }
}

// The adjoint recurrences through one chunk, last step first; writes grad_x
// and accumulates the parameter gradients.  PART: only the first cs steps of
// the chunk are real (cs is wave-uniform; the others are padding and skipped).
template <typename IO, int BL, int L, int V, int CS, bool PART = false, bool ST = false>
__device__ __forceinline__ void reverse_chunk(const BwdArgs& ba, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                              float alpha, float beta_r, int c0, const Stash<BL, CS, V>& st,
                                              const float (&gs)[CS], const float (&gvr)[CS],
                                              BwdLane<IO, BL * kKC<V>>& bl, Accum<BL, BL * kKC<V>>& acc,
                                              int cs = CS) {
  constexpr int KC = kKC<V>, E = BL * KC;
  const ScanArgs& a = ba.s;
  const int64_t rowX = a.N * a.P;
  const float beta = a.beta, vth = a.vth;
#pragma unroll
  for (int k = CS - 1; k >= 0; --k) {
    if (PART && k >= cs) continue;
    const float hk = st.h[k];
    const bool sk = hk >= vth;
    const float sgv = surrogate(hk, vth, kSG<V>, ba.sg_scale);
    const float dS = fmaf(-beta_r * hk, bl.dh_next, gs[k]);  // beta_r = 0: reset detached
    float dh = fmaf(sgv, dS, gvr[k]);
    dh = sk ? dh : fmaf(beta, bl.dh_next, dh);
    // H[t] = beta (1 - S[t-1]) H[t-1] + Z[t]: learnable-beta (PLIF) gradient
    const float hd = k > 0 ? (st.h[k > 0 ? k - 1 : 0] >= vth ? 0.0f : st.h[k > 0 ? k - 1 : 0]) : st.hd0;
    acc.b = fmaf(dh, hd, acc.b);
    float gxo[E];
#pragma unroll
    for (int j = 0; j < BL; ++j) {
      if constexpr (KC == 1) {
        const float tt = kMH<V> ? st.t[kMH<V> ? k : 0][j] : (st.v[k + 1][j] - br.xi[j]) * br.rz[j];
        const float dhk = dh * br.krz[j];
        float y, r;  // psi(u), and r = kappa* dH psi'(u) sgn(Vd - xi) / zeta
        if constexpr (kMH<V>) {
          const float e = st.e[k][j];
          y = st.y[k][j];
          r = (tt * fmaf(2.0f, e, y)) * -dhk;          // psi'(u) sgn = tt (q - 3) e = -tt (y + 2 e)
        } else {
          y = fabsf(tt);
          r = tt > 0.0f ? dhk : (tt < 0.0f ? -dhk : 0.0f);
        }
        bl.lam[j] = kSL<V> ? r : fmaf(alpha, bl.lam[j], r);
        gxo[j] = kRes<V> ? fmaf(dh, br.rp, bl.lam[j]) : bl.lam[j];
        acc.k[j] = fmaf(dh, y, acc.k[j]);
        acc.xi[j] -= r;
        acc.z[j] = fmaf(-r, tt, acc.z[j]);
        if constexpr (!kSL<V>) acc.a = fmaf(bl.lam[j], st.v[k][j], acc.a);
      } else {
        // u = ||d|| rz with d = Vd - xi over the branch's compartments;
        // du/dVd_i = rz d_i / ||d|| (0 at ||d|| = 0), du/dzeta = -u rz.
        const float nrm = __builtin_amdgcn_sqrtf(branch_sumsq<KC>(&st.v[k + 1][j * KC], &br.xi[j * KC]));
        const float u = nrm * br.rz[j];
        const float dhk = dh * br.krz[j];          // kappa* dH / zeta
        float y, w, gzu;  // psi(u), the factor of d_i in dL/dVd_i, and psi'(u) u
        if constexpr (kMH<V>) {
          const float q = u * u;
          const float e = st.e[kMH<V> ? k : 0][j];
          y = fmaf(-q, e, e);                        // (1 - q) e, rounded as in the forward
          const float qe = fmaf(-3.0f, e, q * e);    // psi'(u) / u = (q - 3) e
          w = dhk * (qe * br.rz[j]);                 // kappa* dH psi'(u) rz / ||d||
          gzu = qe * q;
        } else {
          y = u;
          w = nrm > 0.0f ? dhk * __builtin_amdgcn_rcpf(nrm) : 0.0f;
          gzu = u;
        }
#pragma unroll
        for (int i = j * KC; i < (j + 1) * KC; ++i) {
          const float r = w * (st.v[k + 1][i] - br.xi[i]);
          bl.lam[i] = kSL<V> ? r : fmaf(alpha, bl.lam[i], r);
          gxo[i] = kRes<V> ? fmaf(dh, br.rp, bl.lam[i]) : bl.lam[i];
          acc.xi[i] -= r;
          if constexpr (!kSL<V>) acc.a = fmaf(bl.lam[i], st.v[k][i], acc.a);
        }
        acc.k[j] = fmaf(dh, y, acc.k[j]);
        acc.z[j] = fmaf(-dhk, gzu, acc.z[j]);     // -kappa* dH psi'(u) u / zeta
      }
    }
    if constexpr (ST) store_gx_staged<IO, E>(bl.gxbase + int64_t(c0 + k) * rowX, lo.xw, gxo, bl.stage);
    else store_gx<E, kCM<V>>(bl.gxbase + int64_t(c0 + k) * rowX, lo.x, a.xes, gxo);
    bl.dh_next = dh;
  }
}

template <typename IO, int BL, int L, int V, int CS, bool ST = false>
__device__ __forceinline__ void bwd_chunk(const BwdArgs& ba, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                          float alpha, float beta_r, int c0, const float (&v0)[BL * kKC<V>],
                                          float h0, bool s0, const ChunkIn<BL * kKC<V>, CS>& in,
                                          BwdLane<IO, BL * kKC<V>>& bl, Accum<BL, BL * kKC<V>>& acc) {
  Stash<BL, CS, V> st;
  recompute_chunk<BL, L, V, CS>(ba.s, br, alpha, v0, h0, s0, in.x, st);
  reverse_chunk<IO, BL, L, V, CS, false, ST>(ba, lo, br, alpha, beta_r, c0, st, in.gs, in.gv, bl, acc);
}

// Runs the forward from (vd, h, s) at step t_from up to (not including) t_to.
template <typename IO, int BL, int L, int V>
__device__ __forceinline__ void advance(const ScanArgs& a, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                        float alpha, const IO* xbase, int t_from, int t_to,
                                        float (&vd)[BL * kKC<V>], float& h, bool& s) {
  constexpr int E = BL * kKC<V>;
  const int64_t rowX = a.N * a.P;
  for (int t = t_from; t < t_to; ++t) {
    float xv[E];
    load_x<E, kCM<V>>(xbase + int64_t(t) * rowX, lo.x, a.xes, xv);
    const float z = dendrite_step<BL, L, V>(vd, xv, br, alpha);
    soma_step(h, s, z, a.beta, a.vth);
  }
}

// Loads a chunk of CS steps and runs it (used for every chunk but a prefetched one).
template <typename IO, int BL, int L, int V, int CS, bool ST = false>
__device__ __forceinline__ void load_and_run_chunk(const BwdArgs& ba, const LaneOff& lo,
                                                   const Branches<BL, kKC<V>>& br, float alpha, float beta_r,
                                                   int t0, int c0, const SegStart<BL * kKC<V>>& ss,
                                                   BwdLane<IO, BL * kKC<V>>& bl, Accum<BL, BL * kKC<V>>& acc) {
  constexpr int E = BL * kKC<V>;
  ChunkIn<E, CS> in;
  load_chunk_in<IO, E, CS, kCM<V>>(ba.s, lo, bl.xbase, bl.gsbase, bl.gvbase, c0, in);
  float v[E];
#pragma unroll
  for (int j = 0; j < E; ++j) v[j] = ss.v[j];
  float h = ss.h;
  bool s = ss.h >= ba.s.vth && t0 > 0;
  advance<IO, BL, L, V>(ba.s, lo, br, alpha, bl.xbase, t0, c0, v, h, s);
  bwd_chunk<IO, BL, L, V, CS, ST>(ba, lo, br, alpha, beta_r, c0, v, h, s, in, bl, acc);
}

// Chunk plan of a segment [t0, t1): whole KS-step chunks from t0, then the
// remainder in descending powers of two, placed from the top down; visited
// from the last step backwards.  A neuron's first visited chunk is the top of
// its last segment; it is a full KS chunk exactly when that segment's length
// is a multiple of KS, and only then is it prefetched.
template <typename IO, int BL, int L, int V, int KS, bool ST = false>
__device__ __forceinline__ void backward_neuron(const BwdArgs& ba, const LaneOff& lo, int64_t bt,
                                                const Branches<BL, kKC<V>>& br, float alpha,
                                                Accum<BL, BL * kKC<V>>& acc, uint32_t* stage) {
  constexpr int E = BL * kKC<V>;
  const ScanArgs& a = ba.s;
  const int T = int(a.T);
  const int K = a.K;
  const float beta_r = ba.detach ? 0.0f : a.beta;
  const int64_t n0 = bt * a.M;  // first neuron of this batch item (wave-uniform)
  BwdLane<IO, E> bl;
  bl.xbase = static_cast<const IO*>(a.x) + n0 * a.P;
  bl.gxbase = static_cast<IO*>(ba.gx) + n0 * a.P;
  bl.gsbase = static_cast<const IO*>(ba.gspk) + n0;
  bl.gvbase = ba.gv ? ba.gv + n0 : nullptr;
  bl.dh_next = 0.0f;
  bl.stage = stage;
#pragma unroll
  for (int j = 0; j < E; ++j) bl.lam[j] = 0.0f;

  const int nseg = (T + K - 1) / K;
  for (int seg = nseg - 1; seg >= 0; --seg) {
    const int t0 = seg * K;
    const int t1 = min(T, t0 + K);
    SegStart<E> ss;
    load_seg_start<IO, E, kSL<V>>(ba, lo, n0, seg, ss);
    // Chunks: the remainder (len mod KS) first, in descending powers of two
    // from t0, then whole KS-step chunks; visited from the last one back.  A
    // chunk re-runs the forward from t0 up to its first step, so putting the
    // short pieces first keeps that re-advance as short as possible.
    const int len = t1 - t0;
    const int nfull = len / KS;
    const int rem = len - nfull * KS;
    for (int ch = nfull - 1; ch >= 0; --ch) {
      const int c0 = t0 + rem + ch * KS;
      ChunkIn<E, KS> in;
      load_chunk_in<IO, E, KS, kCM<V>>(a, lo, bl.xbase, bl.gsbase, bl.gvbase, c0, in);
      float v[E];
#pragma unroll
      for (int j = 0; j < E; ++j) v[j] = ss.v[j];
      float h = ss.h;
      bool s = ss.h >= a.vth && t0 > 0;
      advance<IO, BL, L, V>(a, lo, br, alpha, bl.xbase, t0, c0, v, h, s);
      bwd_chunk<IO, BL, L, V, KS, ST>(ba, lo, br, alpha, beta_r, c0, v, h, s, in, bl, acc);
    }
    // remainder pieces fill [t0, t0 + rem) with the largest on top and the
    // smallest at t0 (their re-advances then sum to the least); top one first
    int top = t0 + rem;
#pragma unroll
    for (int cs = KS / 2; cs >= 1; cs /= 2) {
      if (rem & cs) {
        const int c0 = top - cs;
        if (cs == 4) load_and_run_chunk<IO, BL, L, V, (KS >= 8 ? 4 : 1), ST>(ba, lo, br, alpha, beta_r, t0, c0, ss, bl, acc);
        else if (cs == 2) load_and_run_chunk<IO, BL, L, V, (KS >= 4 ? 2 : 1), ST>(ba, lo, br, alpha, beta_r, t0, c0, ss, bl, acc);
        else load_and_run_chunk<IO, BL, L, V, 1, ST>(ba, lo, br, alpha, beta_r, t0, c0, ss, bl, acc);
        top = c0;
      }
    }
  }
}

// The common short-sequence case: T == KS, so every neuron is one chunk that
// starts from the zero state.  Software-pipelined over the lane's neurons: the
// next neuron's rows are requested as soon as this neuron's rows are widened to
// float, so they stream in during its recompute and adjoint pass.  FAST: no
// branch of the wave is gated off (no gate select, see recompute_chunk) and no
// grad_v_soma is given (no loads of it).
template <typename IO, int BL, int L, int V, int KS, bool FAST = false, bool ST = false>
__device__ __forceinline__ void single_chunk_items(const BwdArgs& ba, const LaneOff& lo,
                                                   const Branches<BL, kKC<V>>& br, float alpha, int64_t bt0,
                                                   int nk, Accum<BL, BL * kKC<V>>& acc, uint32_t* stage) {
  constexpr int E = BL * kKC<V>;
  const ScanArgs& a = ba.s;
  const float beta_r = ba.detach ? 0.0f : a.beta;
  // The lane's nw positions of each item in turn, then the next item (Walk).
  const Walk wk = make_walk<L, kCM<V>>(a, int64_t(a.ways) * a.M);
  const int nvis = wk.nw * nk;
  int64_t n0 = bt0 * a.M, nx0 = bt0 * a.M * a.P;
  const IO* x = static_cast<const IO*>(a.x);
  const IO* g = static_cast<const IO*>(ba.gspk);
  if (nvis <= 0) return;
  constexpr int W = kRawW<IO, E, kCM<V>>;
  ChunkRaw<IO, E, KS, kCM<V>, ST> cur;
  load_chunk_raw<IO, E, KS, kCM<V>, !FAST, ST>(a, lo, x + nx0, g + n0, ba.gvz + n0, ba.gvn, cur);
  // Every later wait is then counted from loads issued inside the loop, whose
  // next-neuron loads are unconditional (the last neuron runs after it).
  __builtin_amdgcn_s_waitcnt(kWaitVmem);
  int w = 0;
  auto item = [&](const ChunkRaw<IO, E, KS, kCM<V>, ST>& in, bool more, ChunkRaw<IO, E, KS, kCM<V>, ST>& nxt) {
    BwdLane<IO, E> bl;
    bl.stage = stage;
    bl.xbase = x + nx0;
    bl.gxbase = static_cast<IO*>(ba.gx) + nx0;
    bl.gsbase = g + n0;
    bl.gvbase = ba.gv ? ba.gv + n0 : nullptr;
    bl.dh_next = 0.0f;
    float xin[KS][E], gsv[KS], zero[E];
#pragma unroll
    for (int j = 0; j < E; ++j) { bl.lam[j] = 0.0f; zero[j] = 0.0f; }
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      uint32_t raw[W];
      slot_to_lane<W, ST>(in.x[k], stage, raw);
      raw_to_float<IO, E>(raw, xin[k]);
      gsv[k] = raw_to_float<IO>(in.gs[k]);
    }
    float gvv[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) gvv[k] = FAST ? 0.0f : in.gv[k];
    if (more) {
      const bool last_w = ++w == wk.nw;
      if (last_w) w = 0;
      n0 += last_w ? wk.dn_item : wk.dn;
      nx0 += last_w ? wk.dnx_item : wk.dnx;
      load_chunk_raw<IO, E, KS, kCM<V>, !FAST, ST>(a, lo, x + nx0, g + n0, ba.gvz + n0, ba.gvn, nxt);
    }
    // Keeps the requests at this point: left to itself the scheduler sank them
    // below most of the recompute (bf16 layers' backward 2-6 % slower).
    __builtin_amdgcn_sched_barrier(0);
    Stash<BL, KS, V> st;
    recompute_chunk<BL, L, V, KS, FAST>(a, br, alpha, zero, 0.0f, false, xin, st);
    reverse_chunk<IO, BL, L, V, KS, false, ST>(ba, lo, br, alpha, beta_r, 0, st, gsv, gvv, bl, acc);
  };
  for (int i = 0; i + 1 < nvis; ++i) {
    ChunkRaw<IO, E, KS, kCM<V>, ST> nxt;
    item(cur, true, nxt);
    cur = nxt;
  }
  item(cur, false, cur);
}

// The Stateless Dendrite over several checkpoint segments of at most KS steps
// (K <= KS < T).  Its compartments carry no state from step to step, so a
// segment restarts from its checkpointed somatic potential and its own inputs,
// and nothing but dH crosses a segment boundary (in reverse time, within one
// neuron).  Every (neuron, segment) visit is one chunk of KS rows, the rows past
// the segment's end padding (they read one cache line of the segment's first
// row per wave, compute, and are skipped by the adjoint pass).  Software-
// pipelined over the lane's visits like single_chunk_items: the next visit's
// rows and checkpoint are requested right after this visit's recompute, so they
// stream in while its adjoint pass runs.  Visit order: batch items, the lane's
// positions of each item, and each neuron's segments from last to first.
template <typename IO, int E, int CS, bool CM, bool ST = false>
struct SegRaw {
  ChunkRaw<IO, E, CS, CM, ST> in;
  float h0;  // somatic potential before the segment (0 for the first)
};

template <typename IO, int BL, int L, int V, int KS, bool GV = true, bool ST = false>
__device__ __forceinline__ void load_segment_raw(const BwdArgs& ba, const LaneOff& lo, int64_t n0, int64_t nx0,
                                                 int seg, SegRaw<IO, BL * kKC<V>, KS, kCM<V>, ST>& r) {
  constexpr int E = BL * kKC<V>;
  const ScanArgs& a = ba.s;
  const int64_t rowX = a.N * a.P;
  const int T = int(a.T), K = a.K;
  const int c0 = seg * K;
  const int len = min(K, T - c0);
  const IO* x = static_cast<const IO*>(a.x) + nx0;
  const IO* g = static_cast<const IO*>(ba.gspk) + n0;
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const bool real = k < len;
    const int t = real ? c0 + k : c0;
    if constexpr (ST) bload_pieces<kRawW<IO, E, kCM<V>>>(make_rsrc(x + int64_t(t) * rowX), real ? lo.xw : 0u, r.in.x[k]);
    else bload_raw<IO, E, kCM<V>>(make_rsrc(x + int64_t(t) * rowX), real ? lo.x : 0u, a.xes, r.in.x[k]);
    const rsrc_t rg = make_rsrc(g + int64_t(t) * a.N);
    const uint32_t os = real ? lo.s : 0u;
    r.in.gs[k] = sizeof(IO) == 4 ? __builtin_amdgcn_raw_buffer_load_b32(rg, os, 0, kAuxNT)
                                 : uint32_t(__builtin_amdgcn_raw_buffer_load_b16(rg, os, 0, kAuxNT));
    r.in.gv[k] = GV ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                          make_rsrc(ba.gvz + n0 + int64_t(t) * a.N, uniform_u32(real ? ba.gvn : 0u)), lo.v, 0,
                          kAuxNT))
                    : 0.0f;  // GV = false: known absent, nothing is requested
  }
  // checkpointed H after step c0 - 1 (a buffer of no bytes for the first segment)
  const float* hp = seg > 0 ? ba.ckh + int64_t(seg - 1) * a.N + n0 : ba.gvz;
  r.h0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(make_rsrc(hp, uniform_u32(seg > 0 ? 0xFFFFFFFFu : 0u)),
                                                                lo.v, 0, kAuxNT));
}

template <typename IO, int BL, int L, int V, int KS, bool FAST = false, bool ST = false>
__device__ __forceinline__ void stateless_segment_items(const BwdArgs& ba, const LaneOff& lo,
                                                        const Branches<BL, kKC<V>>& br, int64_t bt0, int nk,
                                                        Accum<BL, BL * kKC<V>>& acc, uint32_t* stage) {
  constexpr int E = BL * kKC<V>;
  constexpr int W = kRawW<IO, E, kCM<V>>;
  const ScanArgs& a = ba.s;
  const float beta_r = ba.detach ? 0.0f : a.beta;
  const int T = int(a.T), K = a.K;
  const int nseg = (T + K - 1) / K;
  const Walk wk = make_walk<L, kCM<V>>(a, int64_t(a.ways) * a.M);
  const int nvis = wk.nw * nk * nseg;
  if (nvis <= 0) return;
  // two cursors over the same visit sequence: the visit being loaded, and the
  // one being computed (wave-uniform)
  struct Cursor {
    int64_t n0, nx0;
    int seg, w;
  };
  auto next = [&](Cursor& c) {
    if (c.seg > 0) { --c.seg; return; }
    c.seg = nseg - 1;
    const bool last_w = ++c.w == wk.nw;
    if (last_w) c.w = 0;
    c.n0 += last_w ? wk.dn_item : wk.dn;
    c.nx0 += last_w ? wk.dnx_item : wk.dnx;
  };
  Cursor ld{bt0 * a.M, bt0 * a.M * a.P, nseg - 1, 0};
  Cursor cp = ld;
  SegRaw<IO, E, KS, kCM<V>, ST> cur;
  load_segment_raw<IO, BL, L, V, KS, !FAST, ST>(ba, lo, ld.n0, ld.nx0, ld.seg, cur);
  next(ld);
  // Every later wait is then counted from loads issued inside the loop, whose
  // next-visit loads are unconditional (the last visit runs after it).
  __builtin_amdgcn_s_waitcnt(kWaitVmem);
  BwdLane<IO, E> bl;
  bl.dh_next = 0.0f;
  bl.stage = stage;
  auto visit = [&](const SegRaw<IO, E, KS, kCM<V>, ST>& in, bool more, SegRaw<IO, E, KS, kCM<V>, ST>& nxt) {
    const int c0 = cp.seg * K;
    const int len = min(K, T - c0);
    bl.gxbase = static_cast<IO*>(ba.gx) + cp.nx0;
    if (cp.seg == nseg - 1) bl.dh_next = 0.0f;  // the neuron's last segment: nothing after it
    float xin[KS][E], gsv[KS], zero[E];
#pragma unroll
    for (int j = 0; j < E; ++j) zero[j] = 0.0f;
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      uint32_t raw[W];
      slot_to_lane<W, ST>(in.in.x[k], stage, raw);
      raw_to_float<IO, E>(raw, xin[k]);
      gsv[k] = raw_to_float<IO>(in.in.gs[k]);
    }
    float gvv[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) gvv[k] = FAST ? 0.0f : in.in.gv[k];
    Stash<BL, KS, V> st;
    recompute_chunk<BL, L, V, KS, FAST>(a, br, 0.0f, zero, in.h0, cp.seg > 0 && in.h0 >= a.vth, xin, st);
    if (more) {
      load_segment_raw<IO, BL, L, V, KS, !FAST, ST>(ba, lo, ld.n0, ld.nx0, ld.seg, nxt);
      next(ld);
    }
    reverse_chunk<IO, BL, L, V, KS, true, ST>(ba, lo, br, 0.0f, beta_r, c0, st, gsv, gvv, bl, acc, len);
    next(cp);
  };
  for (int i = 0; i + 1 < nvis; ++i) {
    SegRaw<IO, E, KS, kCM<V>, ST> nxt;
    visit(cur, true, nxt);
    cur = nxt;
  }
  visit(cur, false, cur);
}

// The registers of a stateful wide visit in flight (its X rows and
// checkpointed state travel to LDS): grad_spikes, grad_v_soma and H before the
// segment.
template <int KS>
struct SegSmall {
  uint32_t gs[KS];
  float gv[KS];
  float h0;  // somatic potential before the segment (0 for the first)
};

// Requests visit (n0, nx0, seg): X rows and the checkpointed compartment state
// into `area` (rows past the segment's end are not fetched), the rest into r.
template <typename IO, int BL, int V, int KS, bool FAST>
__device__ __forceinline__ void issue_wide_segment(const BwdArgs& ba, const LaneOff& lo, int64_t n0, int64_t nx0,
                                                   int seg, uint32_t* area, SegSmall<KS>& r) {
  constexpr int W = BL * kKC<V>;
  constexpr int RD = kDmaDw<W>;
  const ScanArgs& a = ba.s;
  const int64_t rowX = a.N * a.P;
  const int T = int(a.T), K = a.K;
  const int c0 = seg * K;
  const int len = min(K, T - c0);
  const IO* x = static_cast<const IO*>(a.x) + nx0;
  const IO* g = static_cast<const IO*>(ba.gspk) + n0;
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const bool real = k < len;
    const int t = real ? c0 + k : c0;
    if (real) dma_pieces<W>(make_rsrc(x + int64_t(t) * rowX), lo.xw, area + k * RD);
    r.gs[k] = __builtin_amdgcn_raw_buffer_load_b32(make_rsrc(g + int64_t(t) * a.N), real ? lo.s : 0u, 0, kAuxNT);
    r.gv[k] = FAST ? 0.0f
                   : __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                         make_rsrc(ba.gvz + n0 + int64_t(t) * a.N, uniform_u32(real ? ba.gvn : 0u)), lo.v, 0,
                         kAuxNT));
  }
  if (seg > 0) dma_pieces<W>(make_rsrc(ba.ckpt + (int64_t(seg - 1) * a.N + n0) * a.P), lo.xw, area + KS * RD);
  const float* hp = seg > 0 ? ba.ckh + int64_t(seg - 1) * a.N + n0 : ba.gvz;
  r.h0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(make_rsrc(hp, uniform_u32(seg > 0 ? 0xFFFFFFFFu : 0u)),
                                                                lo.v, 0, kAuxNT));
}

// The stateful dendrite's wide fp32 lanes (a lane row of more than 16 bytes,
// e.g. ten compartments), every segment one chunk (K <= KS): pipelined over the
// lane's (neuron, segment) visits in the Stateless pipeline's order, but the
// next visit's X rows and checkpointed compartment state travel by LDS DMA
// (dma_pieces) into the wave's LDS area, where they wait without registers:
// the stash of a wide stateful neuron leaves none for rows in flight.  The
// small per-neuron rows (grad_spikes, grad_v_soma, the checkpointed H) ride in
// registers, and grad_x leaves as whole pieces through the wave's `stage`
// buffer (store_gx_staged).  The dendritic adjoint lam and dH cross segment
// boundaries in reverse time within one neuron and restart at its last
// segment.  Rows past a short segment's end are not fetched: the recompute
// runs over whatever the area holds there, and the adjoint pass skips those
// steps.
template <typename IO, int BL, int L, int V, int KS, bool FAST>
__device__ __forceinline__ void stateful_segment_items(const BwdArgs& ba, const LaneOff& lo,
                                                       const Branches<BL, kKC<V>>& br, float alpha, int64_t bt0,
                                                       int nk, Accum<BL, BL * kKC<V>>& acc, uint32_t* area,
                                                       uint32_t* stage) {
  constexpr int E = BL * kKC<V>;
  constexpr int W = E;               // fp32 rows: one dword per compartment
  constexpr int RD = kDmaDw<W>;      // LDS dwords per staged row
  static_assert(sizeof(IO) == 4 && !kSL<V> && !kCM<V>, "stateful wide fp32 lanes only");
  const ScanArgs& a = ba.s;
  const float beta_r = ba.detach ? 0.0f : a.beta;
  const int T = int(a.T), K = a.K;
  const int nseg = (T + K - 1) / K;
  const Walk wk = make_walk<L, kCM<V>>(a, int64_t(a.ways) * a.M);
  const int nvis = wk.nw * nk * nseg;
  if (nvis <= 0) return;
  struct Cursor {
    int64_t n0, nx0;
    int seg, w;
  };
  auto next = [&](Cursor& c) {
    if (c.seg > 0) { --c.seg; return; }
    c.seg = nseg - 1;
    const bool last_w = ++c.w == wk.nw;
    if (last_w) c.w = 0;
    c.n0 += last_w ? wk.dn_item : wk.dn;
    c.nx0 += last_w ? wk.dnx_item : wk.dnx;
  };
  Cursor ld{bt0 * a.M, bt0 * a.M * a.P, nseg - 1, 0};
  Cursor cp = ld;
  SegSmall<KS> cur;
  issue_wide_segment<IO, BL, V, KS, FAST>(ba, lo, ld.n0, ld.nx0, ld.seg, area, cur);
  next(ld);
  BwdLane<IO, E> bl;
  bl.stage = stage;
  bl.dh_next = 0.0f;
  const uint32_t lane = __lane_id();
  for (int i = 0; i < nvis; ++i) {
    const int c0 = cp.seg * K;
    const int len = min(K, T - c0);
    if (cp.seg == nseg - 1) {  // the neuron's last segment: nothing after it
      bl.dh_next = 0.0f;
#pragma unroll
      for (int j = 0; j < E; ++j) bl.lam[j] = 0.0f;
    }
    // this visit's pieces are in the area once every vector memory access of
    // the wave has completed
    __builtin_amdgcn_s_waitcnt(kWaitVmem);
    asm volatile("" ::: "memory");
    float xin[KS][E], v0[E];
#pragma unroll
    for (int k = 0; k < KS; ++k)
#pragma unroll
      for (int j = 0; j < E; ++j) xin[k][j] = __uint_as_float(area[k * RD + lane * W + j]);
    const bool from_ckpt = cp.seg > 0;
#pragma unroll
    for (int j = 0; j < E; ++j) {  // (read unconditionally; the first segment starts from 0)
      const float v = __uint_as_float(area[KS * RD + lane * W + j]);
      v0[j] = from_ckpt ? v : 0.0f;
    }
    float gsv[KS], gvv[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      gsv[k] = __uint_as_float(cur.gs[k]);
      gvv[k] = cur.gv[k];
    }
    const float h0 = cur.h0;
    // the area is refilled only after these reads have completed
    __builtin_amdgcn_s_waitcnt(kWaitLds);
    asm volatile("" ::: "memory");
    if (i + 1 < nvis) {
      issue_wide_segment<IO, BL, V, KS, FAST>(ba, lo, ld.n0, ld.nx0, ld.seg, area, cur);
      next(ld);
    }
    Stash<BL, KS, V> st;
    recompute_chunk<BL, L, V, KS, FAST>(a, br, alpha, v0, h0, from_ckpt && h0 >= a.vth, xin, st);
    bl.gxbase = static_cast<IO*>(ba.gx) + cp.nx0;
    reverse_chunk<IO, BL, L, V, KS, true, true>(ba, lo, br, alpha, beta_r, c0, st, gsv, gvv, bl, acc, len);
    next(cp);
  }
}

// Per channel the backward produces W = 2 B + P parameter gradients, in the
// order g_kappa [B], g_xi [P], g_zeta [B].  Partial slot p of output o of
// channel c lives output-major ([C W][slots], read by one wave per output) when
// there are many slots, slot-major ([slots][C W], one thread per output) when
// there are few.
__device__ __forceinline__ int64_t partial_index(const BwdArgs& ba, int64_t c, int o, int64_t p) {
  const int W = 2 * ba.s.B + ba.s.P;
  const int64_t g = c * W + o;
  return ba.wide ? g * ba.slots + p : p * (ba.s.C * W) + g;
}

// A lane's NV = 2 BL + E accumulators, v = 0 .. NV-1: g_kappa of its BL
// branches, g_xi of its E compartments, g_zeta of its branches.
template <int BL, int E>
__device__ __forceinline__ float accum_value(const Accum<BL, E>& acc, int v) {
  float r = 0.0f;
#pragma unroll
  for (int j = 0; j < BL; ++j) r = v == j ? acc.k[j] : r;
#pragma unroll
  for (int i = 0; i < E; ++i) r = v == BL + i ? acc.xi[i] : r;
#pragma unroll
  for (int j = 0; j < BL; ++j) r = v == BL + E + j ? acc.z[j] : r;
  return r;
}

// Channel output o (0 .. W-1) -> (lane-in-neuron sub, accumulator index v).
template <int BL, int E>
__device__ __forceinline__ void output_source(int o, int B, int P, int* sub, int* v) {
  if (o < B) {
    *sub = o / BL; *v = o % BL;
  } else if (o < B + P) {
    *sub = (o - B) / E; *v = BL + (o - B) % E;
  } else {
    *sub = (o - B - P) / BL; *v = BL + E + (o - B - P) % BL;
  }
}

// Block reduction of the parameter-gradient partials, in a fixed order.
template <int BL, int E, int L>
__device__ __forceinline__ void reduce_partials(const BwdArgs& ba, const Pos& pos, Accum<BL, E>& acc) {
  constexpr int NV = 2 * BL + E;
  const ScanArgs& a = ba.s;
  __shared__ float red[kThreads * E];
  __shared__ float reda[kThreads / 64];
  __shared__ float redb[kThreads / 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int B = a.B, P = a.P, W = 2 * B + P;

  float va = acc.a, vb = acc.b;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    va += __shfl_xor(va, off);
    vb += __shfl_xor(vb, off);
  }
  if (lane == 0) {
    reda[wave] = va;
    redb[wave] = vb;
  }

  if (a.mode == kSpatial) {
    // One channel per block: sum lanes of equal sub within the wave, then waves.
    const int64_t c = pos.c;
    const int64_t jt = pos.tile % a.tpc;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      float x = accum_value(acc, v);
#pragma unroll
      for (int off = 32; off >= L; off >>= 1) x += __shfl_xor(x, off);
      if (lane < L) red[(v * 4 + wave) * L + lane] = x;
    }
    __syncthreads();
    for (int o = tid; o < W; o += kThreads) {
      int sub, v;
      output_source<BL, E>(o, B, P, &sub, &v);
      float sum = 0.0f;
      for (int w = 0; w < 4; ++w) sum += red[(v * 4 + w) * L + sub];
      ba.wsP[partial_index(ba, c, o, int64_t(pos.g) * a.tpc + jt)] = sum;
    }
  } else {
    // Whole channels per tile: sum the batch ways and the S positions of each
    // channel, one accumulator kind (kappa, xi, zeta) at a time.
    for (int q = 0; q < 3; ++q) {
      const int nq = q == 1 ? E : BL;         // accumulators of this kind per lane
      const int v0 = q == 0 ? 0 : (q == 1 ? BL : BL + E);
      const int o0 = q == 0 ? 0 : (q == 1 ? B : B + P);
      const int wq = q == 1 ? P : B;          // outputs of this kind per channel
#pragma unroll
      for (int j = 0; j < E; ++j)
        if (j < nq) red[tid * E + j] = accum_value(acc, v0 + j);
      __syncthreads();
      for (int o = tid; o < a.cpt * wq; o += kThreads) {
        const int slot = o / wq, ol = o % wq;
        const int64_t c = pos.tile * a.cpt + slot;
        if (c >= a.C) continue;
        const int sub = ol / nq, j = ol % nq;
        float sum = 0.0f;
        for (int w = 0; w < a.ways; ++w)
          for (int sp = 0; sp < a.S; ++sp) {
            const int thr = (w * a.pb + slot * int(a.S) + sp) * L + sub;
            sum += red[thr * E + j];
          }
        ba.wsP[partial_index(ba, c, o0 + ol, pos.g)] = sum;
      }
      __syncthreads();
    }
  }
  __syncthreads();
  if (tid == 0) {
    ba.wsA[int64_t(pos.g) * a.ntiles + pos.tile] = (reda[0] + reda[1]) + (reda[2] + reda[3]);
    ba.wsB[int64_t(pos.g) * a.ntiles + pos.tile] = (redb[0] + redb[1]) + (redb[2] + redb[3]);
  }
}

// The backward of the lane's neurons: the short-sequence pipeline (T = KS),
// the Stateless segment pipeline (K <= KS), or neuron by neuron.  ST: wide rows
// staged (see load_pieces; lo.xw is the wave's stretch).
template <typename IO, int BL, int L, int V, int KS, bool ST>
__device__ __forceinline__ void bwd_run(const BwdArgs& ba, const LaneOff& lo, const Branches<BL, kKC<V>>& br,
                                        float alpha, int64_t bt0, int nk, Accum<BL, BL * kKC<V>>& acc,
                                        uint32_t* stage) {
  const ScanArgs& a = ba.s;
  const int T = int(a.T);
  // Without a gated-off branch in the wave (no mask, or a channel whose
  // branches are all on) and without grad_v_soma, the pipelines run a copy
  // without the per-step gate select and without grad_v_soma requests (bf16
  // ImageNet-stem layer: 434 -> 396 VALU instructions per neuron; bf16 backward
  // 1-2 % faster without the empty loads).  The vote is wave-uniform, so each
  // wave runs one copy.
  bool all_on = true;
#pragma unroll
  for (int j = 0; j < BL; ++j) all_on = all_on && br.on[j];
  const bool fast = __all(all_on) && !ba.gv;
  if constexpr (KS == 4) {
    if (T == KS) {
      if (fast) single_chunk_items<IO, BL, L, V, KS, true, ST>(ba, lo, br, alpha, bt0, nk, acc, stage);
      else single_chunk_items<IO, BL, L, V, KS, false, ST>(ba, lo, br, alpha, bt0, nk, acc, stage);
      return;
    }
  }
  if constexpr (kSL<V>) {
    if (a.K <= KS) {
      if (fast) stateless_segment_items<IO, BL, L, V, KS, true, ST>(ba, lo, br, bt0, nk, acc, stage);
      else stateless_segment_items<IO, BL, L, V, KS, false, ST>(ba, lo, br, bt0, nk, acc, stage);
      return;
    }
  }
  for (int i = 0; i < nk; ++i)
    backward_neuron<IO, BL, L, V, KS, false>(ba, lo, bt0 + int64_t(i) * a.ways, br, alpha, acc, stage);
}

template <typename IO, int BL, int L, int V, int KS>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(BL * kKC<V> * KS <= 8 ? 4 : (BL * kKC<V> * KS <= 16 ? 3 : 2)))) dendsn_bwd_kernel(BwdArgs ba) {
  constexpr int E = BL * kKC<V>;
  constexpr int W = kRawW<IO, E, kCM<V>>;
  // Staged wide rows (see load_pieces) for the Stateless Dendrite's pipelines:
  // the stateful dendrite's stash of a wide lane left no room for the pieces
  // (its staged short-sequence copy spilled in the loop).
  constexpr bool kWide = kWideRow<IO, E, kCM<V>> && kSL<V>;
  // The stateful dendrite's wide fp32 lanes move their rows by LDS DMA instead
  // (stateful_segment_items).
  constexpr bool kWideSF = kWideRow<IO, E, kCM<V>> && !kSL<V> && sizeof(IO) == 4;
  if (ba.s.beta_p) ba.s.beta = ba.s.beta_p[0];  // learnable (PLIF) decay
  const ScanArgs& a = ba.s;
  const Pos pos = locate<L>(a);
  const bool full = (kWide || kWideSF) && __all(pos.active);
  Accum<BL, E> acc;
#pragma unroll
  for (int j = 0; j < BL; ++j) acc.k[j] = acc.z[j] = 0.0f;
#pragma unroll
  for (int i = 0; i < E; ++i) acc.xi[i] = 0.0f;
  acc.a = 0.0f;
  acc.b = 0.0f;
  if (pos.active) {
    Branches<BL, kKC<V>> br;
    load_branches<BL, kKC<V>>(a, pos.c, pos.sub, br);
    const float alpha = a.alpha ? a.alpha[0] : 0.0f;
    LaneOff lo = lane_offsets<IO, E, kCM<V>>(a, pos);
    int64_t bt0;
    const int nk = items_of(a, pos, &bt0);
    bool done = false;
    if constexpr (kWide) {
      __shared__ uint32_t stage[kThreads / 64][64 * W];
      lo.xw = __builtin_amdgcn_readfirstlane(lo.x);
      // staged where the loads are too: the two pipelines (the neuron-by-neuron
      // path keeps lane loads and stores)
      const bool pipelined = (KS == 4 && int(a.T) == KS) || a.K <= KS;
      if (full && pipelined && stage_rows<IO>(a, lo.xw, bt0)) {
        bwd_run<IO, BL, L, V, KS, true>(ba, lo, br, alpha, bt0, nk, acc, stage[threadIdx.x >> 6]);
        done = true;
      }
    }
    if constexpr (kWideSF) {
      // one chunk per segment (with T = K = 4 every neuron is one segment:
      // 221 -> 155 us on a T = 4, P = 10 stateful layer against the
      // register-held short-sequence pipeline)
      __shared__ uint32_t area[kThreads / 64][(KS + 1) * kDmaDw<W>];   // rows in flight
      __shared__ uint32_t stage_sf[kThreads / 64][64 * W];              // grad_x leaving
      const uint32_t span = __builtin_amdgcn_readfirstlane(lo.x);
      if (full && a.K <= KS && stage_rows<IO>(a, span, bt0)) {
        lo.xw = span;
        bool all_on = true;  // (as in bwd_run)
#pragma unroll
        for (int j = 0; j < BL; ++j) all_on = all_on && br.on[j];
        if (__all(all_on) && !ba.gv)
          stateful_segment_items<IO, BL, L, V, KS, true>(ba, lo, br, alpha, bt0, nk, acc, area[threadIdx.x >> 6],
                                                          stage_sf[threadIdx.x >> 6]);
        else
          stateful_segment_items<IO, BL, L, V, KS, false>(ba, lo, br, alpha, bt0, nk, acc, area[threadIdx.x >> 6],
                                                           stage_sf[threadIdx.x >> 6]);
        done = true;
      }
    }
    if (!done) bwd_run<IO, BL, L, V, KS, false>(ba, lo, br, alpha, bt0, nk, acc, nullptr);
  }
  if (pos.sub != 0) acc.b = 0.0f;  // the soma runs in every lane of a neuron: count it once
  // every thread of the block reaches this one call (it holds block barriers)
  reduce_partials<BL, E, L>(ba, pos, acc);
}

// Fixed-order float64 sum of the partials into the parameter gradients;
// blocks 0 and 1 reduce g_alpha and g_beta.
__global__ void __launch_bounds__(kThreads) dendsn_finalize_kernel(FinArgs f);

}  // namespace dendsn
