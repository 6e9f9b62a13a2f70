// Device helpers shared by the HIP kernels: bf16 conversion, MFMA operand
// types, raw buffer resources and cache-policy-tagged loads and stores.
#pragma once

#include "spade_internal.h"

#include <math.h>

namespace spade {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;
typedef __amdgpu_buffer_rsrc_t Rsrc;

// sc1 cache policy: a load that sees every device-scope store completed
// before it (it does not hit stale lines of another XCD's L2) and a store that
// writes through to the device coherence point.  Data that one workgroup of a
// persistent launch writes and another reads goes through these.
constexpr int kAuxCoh = 16;
// A byte offset past the end of every buffer resource: loads return 0, stores
// are dropped.  Masks a lane's access without a branch.
constexpr uint32_t kOob = 0x80000000u;

// s_waitcnt that waits until at most N vector-memory operations of this wave
// are outstanding (gfx9 encoding: vmcnt bits [3:0] and [15:14]; expcnt and
// lgkmcnt left at their maxima).  Vector-memory operations complete in issue
// order, so this completes everything issued before the last N.  Direct
// buffer->LDS loads count here; a barrier alone does not wait for them.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// round to nearest even (the hardware conversion, v_cvt_pk_bf16_f32: for
// every non-NaN float the same bits as adding 0x7fff plus the lowest kept
// bit and truncating, checked over all 2^32 inputs); NaN becomes 0x7fc0
__device__ __forceinline__ uint16_t f2bf(float f) {
  if (f != f) return 0x7fc0;
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Raw (unswizzled) buffer resource over [p, p + bytes); bytes < 2^31.
__device__ __forceinline__ Rsrc make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

template <bool COH>
__device__ __forceinline__ uint4 ld_b128(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, COH ? kAuxCoh : 0));
}

// nt cache policy: a streaming read.  With every compute unit streaming lines
// that no other workgroup reads, HBM delivers about 7.0 TB/s with it against
// about 6.1 TB/s without (one to four 8-wave workgroups per CU, plain and
// direct-to-LDS buffer loads alike).  The weight tiles of the verify-call
// GEMMs are loaded with it (each is read by one workgroup, or by the few row
// groups of a wide-row launch, once per call); the big prefill GEMM, whose
// tiles many row-tile workgroups re-read through L2, runs slower with it.
constexpr int kAuxStream = 2;

__device__ __forceinline__ uint4 ld_stream_b128(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kAuxStream));
}

// The same policy for a 16-byte load through a global pointer.
__device__ __forceinline__ uint4 ld_stream_g128(const void* p) {
  typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load((const u32x4*)p));
}

template <bool COH>
__device__ __forceinline__ float ld_f32(Rsrc r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, COH ? kAuxCoh : 0));
}

template <bool COH>
__device__ __forceinline__ float2 ld_f32x2(Rsrc r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, COH ? kAuxCoh : 0);
  return make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
}

template <bool COH>
__device__ __forceinline__ void st_f32(Rsrc r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, COH ? kAuxCoh : 0);
}

template <bool COH>
__device__ __forceinline__ void st_b16(Rsrc r, uint32_t off, uint16_t v) {
  __builtin_amdgcn_raw_buffer_store_b16(v, r, (int)off, 0, COH ? kAuxCoh : 0);
}

// Store v at element `elem` as a GEMM operand: kActSplits bf16 terms
// (hi = rne(v), lo = rne(v - hi), split s at byte s * split_bytes) when the
// weights are bf16, else the float itself.  ok == false drops the store.
template <bool ABF16, bool COH>
__device__ __forceinline__ void st_act(Rsrc r, uint32_t split_bytes, uint32_t elem, bool ok, float v) {
  if constexpr (ABF16) {
    float rem = v;
#pragma unroll
    for (int s = 0; s < kActSplits; ++s) {
      const uint16_t h = f2bf(rem);
      st_b16<COH>(r, ok ? s * split_bytes + elem * 2u : kOob, h);
      rem -= bf2f(h);
    }
  } else {
    st_f32<COH>(r, ok ? elem * 4u : kOob, v);
  }
}

__device__ __forceinline__ float ld_b32_coh(Rsrc r, uint32_t off) { return ld_f32<true>(r, off); }

// buffer resource over memory from `base` on, where base is the same in every
// lane of the wave (offsets are the caller's to keep in bounds)
__device__ __forceinline__ Rsrc wave_rsrc(const void* base) {
  const uint64_t b = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  return make_rsrc((const void*)(((uint64_t)hi << 32) | lo), 0x7ffffff0u);
}

// (max, sum exp(z - max), argmax); ties keep the lower id.
struct RowStat {
  float m, s;
  int a;
};

__device__ __forceinline__ RowStat merge_stat(RowStat x, RowStat y) {
  if (y.m > x.m || (y.m == x.m && y.a < x.a)) {
    const RowStat t = x;
    x = y;
    y = t;
  }
  RowStat o;
  o.m = x.m;
  o.a = x.a;
  o.s = x.s + ((y.m == -INFINITY) ? 0.f : y.s * expf(y.m - x.m));
  return o;
}

__device__ __forceinline__ void flag_error(uint32_t* err, uint32_t bits) {
  if (err) atomicOr(err, bits);
}

}  // namespace spade
