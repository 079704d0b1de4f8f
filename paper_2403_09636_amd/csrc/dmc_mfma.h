// Matrix-core and LDS helpers shared by the gfx950 attention kernels of the
// DMC library (prompt-phase attention and training): direct global-to-LDS
// transfers, v_mfma_f32_32x32x16_bf16 operands, transposed LDS reads and the
// XOR swizzles of the LDS row layouts.  Internal; included by .hip files only.
#pragma once

#include "dmc_device.h"

namespace dmc {
namespace {

constexpr float kLazyRescale = 8.0f;        // log2 of the largest unnormalised probability

// Orders this wave's LDS writes before its later LDS reads (and the reverse).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

template <int CPR>
__device__ __forceinline__ int k_swizzle(int row) { return row & (CPR - 1); }
template <int CPR>
__device__ __forceinline__ int v_swizzle(int row) {
  return CPR == 16 ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
}
__device__ __forceinline__ int vt_swizzle(int dim) { return (dim >> 2) & 3; }
// Rows read both ways (as 16-byte row slices and transposed): for 256-byte
// rows the two 2-bit halves of the row's low nibble are swapped -- distinct
// over any 16 consecutive rows (row reads) and, shifted right by one, over
// any 4 consecutive rows (transposed reads take chunk pairs 2c, 2c + 1).
// Shorter rows keep the value swizzle.
template <int CPR>
__device__ __forceinline__ int dual_swizzle(int row) {
  return CPR == 16 ? (((row & 3) << 2) | ((row >> 2) & 3)) : v_swizzle<CPR>(row);
}
__device__ __forceinline__ int score_slot(int m) {   // pi(m): bits 2 and 3 swapped
  return (m & 0x13) | ((m & 4) << 1) | ((m & 8) >> 1);
}

__device__ __forceinline__ uint32_t lds_offset(const void *p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const char *)p));
}

// Direct global -> LDS transfers: each lane's 16 (or 4, 2) bytes land at
// lds + BYTES * lane, lds wave-uniform (the compiler moves it into m0).  lds
// must point into a __shared__ array: the compiler then knows which array a
// transfer writes and, before each later LDS access of this wave, waits only
// for the transfers into the array accessed (its own vmcnt bookkeeping).  The
// kernels keep every ring slot in an array of its own and issue a fixed
// number of transfers per step (a transfer past the data is switched off,
// not skipped), so that reading one slot does not wait for the transfers in
// flight into the others.  Across waves, completion is awaited explicitly:
// wait_vmcnt, then ring_barrier.  aux carries the cache-policy bits
// (kNontemporal for data streamed once).
constexpr int kCachePolicyDefault = 0;
constexpr int kNontemporal = 2;   // nt (sc0 | nt and sc1 | nt measured the same)
constexpr uint32_t kOutOfRange = 0x80000000u;   // a lane offset past every buffer range

typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(1))) char global_cchar_t;

// Per-lane 64-bit global addresses (the compiler cannot attribute these to
// a slot as precisely; used where every transfer is awaited before the LDS
// is read).
template <int AUX = kCachePolicyDefault>
__device__ __forceinline__ void dma16(void *lds, const void *g) {
  __builtin_amdgcn_global_load_lds((global_cchar_t *)g, (lds_void_t *)lds, 16, 0, AUX);
}

// A wave-uniform 64-bit base (SGPRs, see uniform_ptr) and a 32-bit per-lane
// offset, by the buffer form of the transfer: the base goes into a raw
// buffer resource (stride 0, range 2^31 - 1 bytes, or 0 when the transfer is
// off: then every lane is out of range and nothing is read).  A lane offset
// of kOutOfRange switches that lane off alone.  Out-of-range lanes read no
// memory; what their LDS bytes then hold is not relied upon.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const char *sbase, bool on = true) {
  // on is wave-uniform: made visibly so, else the compiler loops over lanes
  const int range = __builtin_amdgcn_readfirstlane(on ? 0x7fffffff : 0);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(sbase), static_cast<short>(0), range,
                                           0x00020000);
}
template <int AUX = kCachePolicyDefault, int BYTES = 16>
__device__ __forceinline__ void dma_so(void *lds, const char *sbase, uint32_t voff, bool on = true) {
  static_assert(BYTES == 16 || BYTES == 4 || BYTES == 2, "transfer width");
  if constexpr (BYTES == 16)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(raw_rsrc(sbase, on), (lds_void_t *)lds, 16, voff, 0, 0,
                                             AUX);
  else if constexpr (BYTES == 4)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(raw_rsrc(sbase, on), (lds_void_t *)lds, 4, voff, 0, 0,
                                             AUX);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(raw_rsrc(sbase, on), (lds_void_t *)lds, 2, voff, 0, 0,
                                             AUX);
}
__device__ __forceinline__ void dma16_s(void *lds, const char *sbase, uint32_t voff, bool on = true) {
  dma_so<kCachePolicyDefault>(lds, sbase, voff, on);
}

// dma16_s with the nontemporal policy, for data streamed once (no reuse
// through the caches).
__device__ __forceinline__ void dma16_s_nt(void *lds, const char *sbase, uint32_t voff,
                                           bool on = true) {
  dma_so<kNontemporal>(lds, sbase, voff, on);
}

// Workgroup barrier of the block rings.  This wave's LDS reads and writes
// are complete before it (lgkmcnt(0)) and none moves across it (compiler
// fences), but transfers still in flight into other ring slots are not
// awaited: the release fence of __syncthreads would wait for every
// outstanding global -> LDS transfer of the wave.  Every wave awaits its own
// transfers into the slot that is read next (wait_vmcnt) before the barrier.
__device__ __forceinline__ void ring_barrier() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0) only
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// The one-wave counterpart: this wave's LDS reads and writes are complete
// (lgkmcnt(0)) and none moves across it, without a wait for transfers.  The
// compiler waits for a transfer before reading its array, but it does not
// order a transfer after earlier reads of the same array: a slot is refilled
// only after this sync (a transfer that is switched off, or served from a
// cache, can land within cycles).
__device__ __forceinline__ void wave_ring_sync() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0) only
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// A wave-uniform pointer, made visibly uniform (SGPRs) for dma16_s.
__device__ __forceinline__ const char *uniform_ptr(const char *ptr) {
  const uint64_t x = reinterpret_cast<uint64_t>(ptr);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x >> 32));
  return reinterpret_cast<const char *>((uint64_t(hi) << 32) | lo);
}

// s_waitcnt with only the vector-memory count (at most N outstanding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint2 ds_read_tr16(const void *p) {
  const bf16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4_t *)((__attribute__((address_space(3))) char *)p));
  return __builtin_bit_cast(uint2, v);
}

__device__ __forceinline__ f32x16_t mfma_32x32x16(const uint4 &a, const uint4 &b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Maximum of x over lanes l and l ^ 32 (v_permlane32_swap of x with itself
// leaves each lane's value and its partner's in the two results).
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                  __builtin_bit_cast(unsigned, x), false, false);
  return fmaxf(__builtin_bit_cast(float, static_cast<unsigned>(r[0])),
               __builtin_bit_cast(float, static_cast<unsigned>(r[1])));
}

// Maximum of x over lanes l and l ^ 16 (v_permlane16_swap of x with itself
// leaves rows 0/2 in one result and rows 1/3 in the other).  No LDS access.
__device__ __forceinline__ float max_rows16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x),
                                                  __builtin_bit_cast(unsigned, x), false, false);
  return fmaxf(__builtin_bit_cast(float, static_cast<unsigned>(r[0])),
               __builtin_bit_cast(float, static_cast<unsigned>(r[1])));
}

// Two floats -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  typedef float f2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 b2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2_t{lo, hi}, b2_t));
}

// Sum of a packed bf16 pair added to acc (exact products by 1, fp32 sum).
__device__ __forceinline__ float add_pair(uint32_t pair, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pair),
                                         __builtin_bit_cast(bf16x2_t, 0x3f803f80u), acc, false);
}

}  // namespace
}  // namespace dmc
