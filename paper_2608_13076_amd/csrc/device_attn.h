// Verify attention for a bf16 cache with head_dim 128 (Sec. III-A: the
// gamma+1 appended rows of a request attend causally to its cached keys and
// to each other).
//
// Work item: (request, head, chunk of CK keys), one 8-wave workgroup.  Row i
// of the request sits at position L + i and sees keys <= L + i.  Scores
// S = Q K^T run with keys split over the waves (wave w: keys
// [k_lo + w CK/8, k_lo + (w+1) CK/8)); the chunk softmax runs one wave per
// row; O = P V runs with features split over the waves (wave w: features
// [16 w, 16 w + 16) over every key of the chunk), so each wave ends with
// final chunk outputs and no cross-wave sum is needed.  Both products use
// MFMA 16x16x32 bf16 with Q and P split into two bf16 terms (hi + lo).  K and
// V are stored in blocks of 256 positions in the order of the B operands of
// S = Q K^T and O = P V (k_cache_index, v_cache_index), so every B-operand
// fragment a wave loads is 1 KB contiguous.  A chunk writes its unnormalised output, row
// max and row sum; the chunks of a (request, head) are merged in chunk order
// with weights exp(m_c - max) / sum_c(l_c exp(m_c - max)).
#pragma once

#include "device_util.h"

namespace spade {

constexpr int kAttnRows = 16;  // rows per request (gamma + 1 <= 16)
constexpr int kAttnThreads = 512;

template <int CK>
struct AttnSmem {
  static_assert(CK == 128 || CK == 256, "chunk of 128 or 256 keys");
  // probabilities as two bf16 terms (the A operand of O = P V); rows padded by
  // 16 bytes so the 16 rows of a fragment read start in different banks; 16-byte
  // aligned, so each lane's fragment is one ds_read_b128 (with the alignment of
  // uint16_t alone it becomes two ds_read2_b32, whose 64 lanes conflict)
  alignas(16) uint16_t ph[kAttnRows][CK + 8];
  alignas(16) uint16_t pl[kAttnRows][CK + 8];
  float pm[kAttnRows][8], ps[kAttnRows][8];  // per-wave row max / row sum
  float m[kAttnRows], l[kAttnRows];
};

template <int CK>
struct AttnRegs {
  uint4 kf[CK / 128][4];  // [16-key group][32-feature slice]: key k_lo + (CK/8) w + 16 grp + kl
  uint4 vf[CK / 32];      // [32-key step]: V^T row 16 w + kl, keys k_lo + 32 ks + 8 g .. + 8
};

struct AttnItem {
  bool active;
  int bl, h, c;
  int L;           // cached keys of the request (row i sits at L + i)
  int nc;          // chunks of the request
  int k_lo, k_hi;  // keys of this chunk: [k_lo, k_hi)
  const uint16_t* kc;  // K blocks of (request, head) (k_cache_index)
  const uint16_t* vc;  // V^T rows of (request, head)
};

// Item (request bl, head h, chunk c) of a request with L cached keys and R
// rows; chunks at or past the request's last key are inactive.
template <int CK>
__device__ __forceinline__ AttnItem attn_item(bool valid, int bl, int h, int c, int L, int R, const void* kc,
                                              const void* vc, size_t head_off) {
  AttnItem it;
  it.bl = bl;
  it.h = h;
  it.c = c;
  it.L = L;
  it.nc = (L + R + CK - 1) / CK;
  it.active = valid && c < it.nc;
  it.k_lo = c * CK;
  it.k_hi = it.active ? min(it.k_lo + CK, L + R) : it.k_lo;
  it.kc = (const uint16_t*)kc + head_off;
  it.vc = (const uint16_t*)vc + head_off;
  return it;
}

// Zero the V^T entries of keys at or past k_hi (their P is zero, but the
// cache may hold anything there).
template <int CK>
__device__ __forceinline__ void attn_mask_tail(const AttnItem& it, int lane, AttnRegs<CK>& r) {
  const int g = lane >> 4;
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const int kv0 = it.k_lo + 32 * ks + 8 * g;
    if (kv0 + 8 > it.k_hi) {
      uint32_t w[4] = {r.vf[ks].x, r.vf[ks].y, r.vf[ks].z, r.vf[ks].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int p0 = kv0 + 2 * e;
        if (p0 >= it.k_hi) w[e] = 0u;
        else if (p0 + 1 >= it.k_hi) w[e] &= 0xffffu;
      }
      r.vf[ks] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// f2bf without the NaN canonicalisation (the probabilities of a chunk are
// NaN only when its scores are, and then the outputs are NaN either way).
__device__ __forceinline__ uint16_t f2bf_num(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

__device__ __forceinline__ void attn_split2(const float* xs, uint4& hi, uint4& lo) {
  uint32_t hw[4], lw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint16_t h0 = f2bf(xs[2 * e]), h1 = f2bf(xs[2 * e + 1]);
    const uint16_t l0 = f2bf(xs[2 * e] - bf2f(h0)), l1 = f2bf(xs[2 * e + 1] - bf2f(h1));
    hw[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    lw[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = make_uint4(hw[0], hw[1], hw[2], hw[3]);
  lo = make_uint4(lw[0], lw[1], lw[2], lw[3]);
}

// Queries staged in LDS as their two bf16 terms (rows of kAttnQPitch
// elements: 16-byte aligned, consecutive rows four banks apart).  Four
// consecutive features x of row `row` go in as attn_split2 splits them.
constexpr int kAttnQPitch = kAttnHd + 8;

__device__ __forceinline__ void attn_stage_q(uint16_t (*sqh)[kAttnQPitch], uint16_t (*sql)[kAttnQPitch], int row,
                                             int f, float4 x) {
  const float xs[4] = {x.x, x.y, x.z, x.w};
  uint32_t hw[2], lw[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const uint16_t h0 = f2bf(xs[2 * e]), h1 = f2bf(xs[2 * e + 1]);
    const uint16_t l0 = f2bf(xs[2 * e] - bf2f(h0)), l1 = f2bf(xs[2 * e + 1] - bf2f(h1));
    hw[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    lw[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  *(uint2*)&sqh[row][f] = make_uint2(hw[0], hw[1]);
  *(uint2*)&sql[row][f] = make_uint2(lw[0], lw[1]);
}

// Cross-lane moves within a row of 16 lanes (DPP): lane i reads lane i^1,
// i^2, 7-i (within its half row) and 15-i; the four steps reduce the row.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_f32<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_f32<0x141>(v));  // row_half_mirror
  return fmaxf(v, dpp_f32<0x140>(v));  // row_mirror
}

__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x141>(v);
  return v + dpp_f32<0x140>(v);
}

// One chunk of the verify attention: the K fragments come from attn_load_k,
// the queries from LDS (sqh / sql, their bf16 terms staged by the caller with
// attn_stage_q: row i, feature f at [i][f], rows past R zero), and the V^T
// fragments are requested only after the score products, into the registers
// the K fragments held, so a wave holds one of the two at a time.
//
// Chunk softmax: each lane holds the scores of rows 4g..4g+3 for its keys;
// row maxima and sums reduce over the 16 lanes of a row (DPP) and then over
// the eight waves (LDS, in wave order).  Probabilities (exp2 of the
// log2(e)-scaled difference) go to LDS once, as two bf16 terms, and every
// wave reads them as the A operand of O = P V.
template <int CK>
__device__ __forceinline__ void attn_load_k(const AttnItem& it, int wave, int lane, uint4 (&kf)[CK / 128][4]) {
  const int g = lane >> 4, kl = lane & 15;
#pragma unroll
  for (int grp = 0; grp < CK / 128; ++grp) {
    const int key = it.k_lo + (CK / 8) * wave + 16 * grp + kl;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) kf[grp][ks] = make_uint4(0, 0, 0, 0);
    if (key < it.k_hi) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) kf[grp][ks] = ld_stream_g128(it.kc + k_cache_index(32 * ks + 8 * g, key, kAttnHd));
    }
  }
}

// Scores of one chunk, scaled and masked: sv[grp][i] is row 4g + i and key
// k_lo + (CK/8) wave + 16 grp + kl of the lane (-inf past k_hi or after the
// row's position).
template <int CK>
__device__ __forceinline__ void attn_scores(const AttnItem& it, const uint4 (&kf)[CK / 128][4],
                                            const uint16_t (*sqh)[kAttnQPitch], const uint16_t (*sql)[kAttnQPitch],
                                            float scale, float (&sv)[CK / 128][4]) {
  constexpr int NG = CK / 128;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
#pragma unroll
  for (int grp = 0; grp < NG; ++grp) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 qh = *(const uint4*)&sqh[kl][32 * ks + 8 * g];
      const uint4 ql = *(const uint4*)&sql[kl][32 * ks + 8 * g];
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ql),
                                                    __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qh),
                                                    __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
    }
    const int key = it.k_lo + (CK / 8) * wave + 16 * grp + kl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * g + i;
      sv[grp][i] = (key < it.k_hi && key <= it.L + row) ? acc[i] * scale : -INFINITY;
    }
  }
}

// V^T fragments of a chunk: 8-key granules below k_hi rounded up to 8 (zero
// past them).  A chunk's keys lie in one V block, where the fragment of
// (feature tile = wave, 32-key step) is 1 KB contiguous (v_cache_index).
template <int CK>
__device__ __forceinline__ void attn_load_v(const AttnItem& it, int wave, int lane, AttnRegs<CK>& r) {
  static_assert(kVBlock % CK == 0, "a chunk within one V block");
  const int g = lane >> 4, kl = lane & 15;
  const int ke = (it.k_hi + 7) & ~7;
  const uint16_t* vfr = it.vc + v_cache_index(16 * wave + kl, it.k_lo + 8 * g, kAttnHd);
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const int kv0 = it.k_lo + 32 * ks + 8 * g;
    r.vf[ks] = make_uint4(0, 0, 0, 0);
    if (kv0 + 8 <= ke) r.vf[ks] = ld_stream_g128(vfr + ks * 512);
  }
}

// Chunk softmax of the scores: probabilities to sm.ph / sm.pl, and the row
// max and row sum of rows < R to sm.m / sm.l (read after a barrier).
template <int CK>
__device__ __forceinline__ void attn_softmax(const float (&sv)[CK / 128][4], int R, AttnSmem<CK>& sm) {
  constexpr int NG = CK / 128;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float mx = sv[0][i];
#pragma unroll
    for (int grp = 1; grp < NG; ++grp) mx = fmaxf(mx, sv[grp][i]);
    mx = row16_max(mx);
    if (kl == 0) sm.pm[4 * g + i][wave] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * g + i;
    const float4 a = *(const float4*)&sm.pm[row][0];
    const float4 b = *(const float4*)&sm.pm[row][4];
    const float M = fmaxf(fmaxf(fmaxf(a.x, a.y), fmaxf(a.z, a.w)), fmaxf(fmaxf(b.x, b.y), fmaxf(b.z, b.w)));
    float sum = 0.f;
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      const float e = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((sv[grp][i] - M) * 1.44269504088896341f);
      sum += e;
      const uint16_t h = f2bf_num(e);
      const int kc = (CK / 8) * wave + 16 * grp + kl;
      sm.ph[row][kc] = h;
      sm.pl[row][kc] = f2bf_num(e - bf2f(h));
    }
    sum = row16_sum(sum);
    if (kl == 0) sm.ps[row][wave] = sum;
  }
  __syncthreads();
  if (tid < R) {
    float l = 0.f, M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      l += sm.ps[tid][w];
      M = fmaxf(M, sm.pm[tid][w]);
    }
    sm.m[tid] = M;
    sm.l[tid] = l;
  }
}

// O = P V over the chunk (P from sm.ph / sm.pl, V^T fragments masked past
// k_hi): row 4g + i, feature 16 wave + kl in o[i].
template <int CK>
__device__ __forceinline__ floatx4 attn_pv(const AttnSmem<CK>& sm, const AttnRegs<CK>& r) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, kl = lane & 15;
  floatx4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const uint4 ph = *(const uint4*)&sm.ph[kl][32 * ks + 8 * g];
    const uint4 pl = *(const uint4*)&sm.pl[kl][32 * ks + 8 * g];
    o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pl), __builtin_bit_cast(bf16x8, r.vf[ks]), o,
                                                0, 0, 0);
    o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ph), __builtin_bit_cast(bf16x8, r.vf[ks]), o,
                                                0, 0, 0);
  }
  return o;
}

// The verify kernels' chunk: the helpers above written out in one body, the
// same operations in the same order (composed of the helper calls, the
// one-chunk kernel needs 80 VGPRs and spills six; written out, 76 and none).
template <int CK>
__device__ __forceinline__ floatx4 attn_chunk_lr(const AttnItem& it, const uint4 (&kf)[CK / 128][4],
                                                 const uint16_t (*sqh)[kAttnQPitch],
                                                 const uint16_t (*sql)[kAttnQPitch], int R, float scale,
                                                 AttnSmem<CK>& sm) {
  constexpr int NG = CK / 128;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
  const int ke = (it.k_hi + 7) & ~7;
  float sv[NG][4];
#pragma unroll
  for (int grp = 0; grp < NG; ++grp) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 qh = *(const uint4*)&sqh[kl][32 * ks + 8 * g];
      const uint4 ql = *(const uint4*)&sql[kl][32 * ks + 8 * g];
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ql),
                                                    __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qh),
                                                    __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
    }
    const int key = it.k_lo + (CK / 8) * wave + 16 * grp + kl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * g + i;
      sv[grp][i] = (key < it.k_hi && key <= it.L + row) ? acc[i] * scale : -INFINITY;
    }
  }
  // the V^T fragments, after the score products (the K registers are free);
  // fragment (wave, 32-key step ks) of the chunk's V block is 512 elements
  // after step ks - 1's
  __builtin_amdgcn_sched_barrier(0);
  AttnRegs<CK> r;
  const uint16_t* vfr = it.vc + v_cache_index(16 * wave + kl, it.k_lo + 8 * g, kAttnHd);
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const int kv0 = it.k_lo + 32 * ks + 8 * g;
    r.vf[ks] = make_uint4(0, 0, 0, 0);
    if (kv0 + 8 <= ke) r.vf[ks] = ld_stream_g128(vfr + ks * 512);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float mx = sv[0][i];
#pragma unroll
    for (int grp = 1; grp < NG; ++grp) mx = fmaxf(mx, sv[grp][i]);
    mx = row16_max(mx);
    if (kl == 0) sm.pm[4 * g + i][wave] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * g + i;
    const float4 a = *(const float4*)&sm.pm[row][0];
    const float4 b = *(const float4*)&sm.pm[row][4];
    const float M = fmaxf(fmaxf(fmaxf(a.x, a.y), fmaxf(a.z, a.w)), fmaxf(fmaxf(b.x, b.y), fmaxf(b.z, b.w)));
    float sum = 0.f;
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      const float e = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((sv[grp][i] - M) * 1.44269504088896341f);
      sum += e;
      const uint16_t h = f2bf_num(e);
      const int kc = (CK / 8) * wave + 16 * grp + kl;
      sm.ph[row][kc] = h;
      sm.pl[row][kc] = f2bf_num(e - bf2f(h));
    }
    sum = row16_sum(sum);
    if (kl == 0) sm.ps[row][wave] = sum;
  }
  __syncthreads();
  if (tid < R) {
    float l = 0.f, M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      l += sm.ps[tid][w];
      M = fmaxf(M, sm.pm[tid][w]);
    }
    sm.m[tid] = M;
    sm.l[tid] = l;
  }
  attn_mask_tail(it, lane, r);
  floatx4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const uint4 ph = *(const uint4*)&sm.ph[kl][32 * ks + 8 * g];
    const uint4 pl = *(const uint4*)&sm.pl[kl][32 * ks + 8 * g];
    o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pl), __builtin_bit_cast(bf16x8, r.vf[ks]), o,
                                                0, 0, 0);
    o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ph), __builtin_bit_cast(bf16x8, r.vf[ks]), o,
                                                0, 0, 0);
  }
  return o;
}

// Last-arrival merge of the chunks of one (request, head).
struct AttnMergeSmem {
  float sc[kAttnMaxChunks][kAttnRows];  // merge weights
  int last;
};

// partials of output o (= row * kAttnHd + dd) for chunks c0 .. c0 + 15
// (COH: sc1 loads; chunks past nc and ok == false read 0)
template <bool COH>
__device__ __forceinline__ void attn_load16(Rsrc rpo, int c0, int nc, int Rmax, int o, bool ok, float (&v)[16]) {
  const int row = o / kAttnHd, dd = o - row * kAttnHd;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int c = c0 + j;
    v[j] = ld_f32<COH>(rpo, (ok && c < nc) ? (uint32_t)((c * Rmax + row) * kAttnHd + dd) * 4u : kOob);
  }
}

// One chunk's term of a merged output: O + w v (a zero weight adds zero
// whatever v holds), rounded after the product and after the sum, never
// fused, so every merge gives the same bits.
__device__ __forceinline__ float attn_acc1(float O, float v, float w) {
#pragma clang fp contract(off)
  return O + (w != 0.f ? v * w : 0.f);
}

// add chunks c0 .. c0 + 15 of output o to O, in chunk order
__device__ __forceinline__ void attn_acc16(const AttnMergeSmem& ms, int c0, int nc, int o, const float (&v)[16],
                                           float& O) {
  const int row = o / kAttnHd;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int c = c0 + j;
    if (c < nc) O = attn_acc1(O, v[j], ms.sc[c][row]);
  }
}

// merged outputs oa and oa + 512 (each where < nout); va / vb hold their
// chunks 0..15 on entry
template <bool COH, class Out>
__device__ __forceinline__ void attn_merge_pair(Rsrc rpo, const AttnMergeSmem& ms, int nc, int Rmax, int nout,
                                                int oa, float (&va)[16], float (&vb)[16], Out&& out) {
  const int ob = oa + 512;
  float Oa = 0.f, Ob = 0.f;
  attn_acc16(ms, 0, nc, oa, va, Oa);
  attn_acc16(ms, 0, nc, ob, vb, Ob);
  for (int c0 = 16; c0 < nc; c0 += 16) {
    attn_load16<COH>(rpo, c0, nc, Rmax, oa, oa < nout, va);
    attn_load16<COH>(rpo, c0, nc, Rmax, ob, ob < nout, vb);
    attn_acc16(ms, c0, nc, oa, va, Oa);
    attn_acc16(ms, c0, nc, ob, vb, Ob);
  }
  if (oa < nout) out(oa, Oa);
  if (ob < nout) out(ob, Ob);
}

// Publish this chunk's partial (o: the chunk function's result) with write-through
// stores, arrive on the counter of its (request, head) once the stores have
// landed, and, in the workgroup that arrives last, merge the request's
// chunks and pass each merged output o = row * kAttnHd + dd to out(o, value).
// Merge weights of a row: one wave, chunks over its lanes; the weight of
// chunk c is exp(m_c - max) / sum_c(l_c exp(m_c - max)).  The last arrival
// resets the counter.  part_o / part_ml: [bh][NC][Rmax][kAttnHd] /
// [bh][NC][Rmax][2].  All 512 threads call it; inactive items only
// synchronise.
// Store this chunk's partial (o: the chunk function's result; m / l from sa) with
// write-through stores, without waiting for them.
template <int CK>
__device__ __forceinline__ void attn_publish(const AttnItem& it, floatx4 o, const AttnSmem<CK>& sa, float* part_o,
                                             float* part_ml, int H, int NC, int Rmax, int R) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
  const size_t bh = (size_t)it.bl * H + it.h;
  if (it.active) {
    float* po = part_o + ((bh * NC + it.c) * Rmax) * kAttnHd + 16 * wave + kl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * g + i;
      if (row < R) __hip_atomic_store(po + row * kAttnHd, o[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    float* pml = part_ml + ((bh * NC + it.c) * Rmax) * 2;
    if (tid < R) {
      __hip_atomic_store(pml + tid * 2, sa.m[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(pml + tid * 2 + 1, sa.l[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Merge weights of one row's nc chunks, by one wave (chunk c on lane c % 64,
// slot c / 64): w_c = exp(m_c - max) / sum_c(l_c exp(m_c - max)), the sum
// taken per lane in slot order and then across the lanes by butterfly.
// ml(c, ok, m, l) fetches chunk c's row max and row sum (ok false: no such
// chunk, values unused); put(c, w) receives each weight after every fetch.
template <class ML, class PUT>
__device__ __forceinline__ void attn_row_weights(int nc, ML&& ml, PUT&& put) {
  const int lane = threadIdx.x & 63;
  constexpr int NJ = kAttnMaxChunks / 64;
  float mc[NJ], lc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = lane + 64 * j;
    const bool ok = c < nc;
    float m, l;
    ml(c, ok, m, l);
    mc[j] = ok ? m : -INFINITY;
    lc[j] = l;
  }
  float Mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < NJ; ++j) Mx = fmaxf(Mx, mc[j]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) Mx = fmaxf(Mx, __shfl_xor(Mx, off));
  float Ls = 0.f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    mc[j] = (mc[j] == -INFINITY) ? 0.f : expf(mc[j] - Mx);
    Ls += lc[j] * mc[j];
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) Ls += __shfl_xor(Ls, off);
  const float inv = 1.0f / Ls;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = lane + 64 * j;
    if (c < nc) put(c, mc[j] * inv);
  }
}

// Merge weights of the nc chunks of R rows into ms.sc (attn_row_weights, one
// wave per row: rows wave and wave + 8); ml(c, row, ok, m, l) as there.  All
// 512 threads call it; the caller synchronises before reading ms.sc.
template <class ML>
__device__ __forceinline__ void attn_merge_weights(AttnMergeSmem& ms, int nc, int R, ML&& ml) {
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int row = wave + 8 * k;
    if (row < R)  // uniform across the wave
      attn_row_weights(
          nc, [&](int c, bool ok, float& m, float& l) { ml(c, row, ok, m, l); },
          [&](int c, float w) { ms.sc[c][row] = w; });
  }
}

// Merge the nc chunk partials of (request, head) bh in chunk order and pass
// each merged output o = row * kAttnHd + dd to out(o, value).  Merge weights
// of a row: one wave, chunks over its lanes; the weight of chunk c is
// exp(m_c - max) / sum_c(l_c exp(m_c - max)).  All 512 threads call it.
template <bool COH, class Out>
__device__ __forceinline__ void attn_merge(size_t bh, int nc, AttnMergeSmem& ms, float* part_o, float* part_ml,
                                           int NC, int Rmax, int R, Out&& out) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // this thread's first partials, and the (m, l) pairs of the wave's rows
  // (wave and wave + 8: R <= 16), in one round trip
  const Rsrc rpo = wave_rsrc(part_o + (bh * NC * Rmax) * kAttnHd);
  const Rsrc rpm = wave_rsrc(part_ml + (bh * NC * Rmax) * 2);
  const int nout = R * kAttnHd;
  float va[16], vb[16];
  attn_load16<COH>(rpo, 0, nc, Rmax, tid, tid < nout, va);
  attn_load16<COH>(rpo, 0, nc, Rmax, tid + 512, tid + 512 < nout, vb);
  attn_merge_weights(ms, nc, R, [&](int c, int row, bool ok, float& m, float& l) {
    const uint32_t off = ok ? (uint32_t)((c * Rmax + row) * 2) * 4u : kOob;
    m = ld_f32<COH>(rpm, off);
    l = ld_f32<COH>(rpm, off == kOob ? kOob : off + 4u);
  });
  __syncthreads();
  attn_merge_pair<COH>(rpo, ms, nc, Rmax, nout, tid, va, vb, out);
  for (int oa = tid + 1024; oa < nout; oa += 1024) {
    attn_load16<COH>(rpo, 0, nc, Rmax, oa, true, va);
    attn_load16<COH>(rpo, 0, nc, Rmax, oa + 512, oa + 512 < nout, vb);
    attn_merge_pair<COH>(rpo, ms, nc, Rmax, nout, oa, va, vb, out);
  }
}

// Once this workgroup's published partials (n_mine chunks of the (request,
// head) of it) have landed, arrive on the counter of that (request, head)
// with n_mine, and, in the workgroup whose arrival completes the request's
// chunks, merge them and pass each merged output o = row * kAttnHd + dd to
// out(o, value).  The completing arrival resets the counter.  All 512 threads
// call it.  COH: read the partials with sc1 loads; without it they are read
// with plain loads, which is enough within one launch (no workgroup of the
// launch reads a partial before its write-through store has landed, and the
// launch starts with the L2 invalidated).
template <bool COH = true, class Out>
__device__ __forceinline__ void attn_arrive_merge(const AttnItem& it, int n_mine, AttnMergeSmem& ms, float* part_o,
                                                  float* part_ml, uint32_t* attn_cnt, int H, int NC, int Rmax, int R,
                                                  Out&& out) {
  const int tid = threadIdx.x;
  const size_t bh = (size_t)it.bl * H + it.h;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) {
    int last = 0;
    if (n_mine > 0) {
      uint32_t* cnt = attn_cnt + bh;
      const uint32_t old = __hip_atomic_fetch_add(cnt, (uint32_t)n_mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (old + (uint32_t)n_mine == (uint32_t)it.nc) {
        __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = 1;
      }
    }
    ms.last = last;
  }
  __syncthreads();
  if (!ms.last) return;  // uniform across the workgroup
  attn_merge<COH>(bh, it.nc, ms, part_o, part_ml, NC, Rmax, R, out);
}

// attn_publish and attn_arrive_merge for a workgroup that computed the one
// chunk it.
template <int CK, bool COH = true, class Out>
__device__ __forceinline__ void attn_publish_merge(const AttnItem& it, floatx4 o, const AttnSmem<CK>& sa,
                                                   AttnMergeSmem& ms, float* part_o, float* part_ml,
                                                   uint32_t* attn_cnt, int H, int NC, int Rmax, int R, Out&& out) {
  attn_publish<CK>(it, o, sa, part_o, part_ml, H, NC, Rmax, R);
  attn_arrive_merge<COH>(it, it.active ? 1 : 0, ms, part_o, part_ml, attn_cnt, H, NC, Rmax, R, out);
}

// Grouped-query variant of attn_chunk_lr: one workgroup computes the chunk
// for all G query heads of a K/V head, so the chunk's keys and values pass
// through the compute unit once.  The G R rows are packed into T 16-row
// tiles (packed row pr = gg R + i: query head gg of the group, request row
// i; rows past G R are masked).  Every packed row goes through the same
// instructions in the same order as its row in attn_chunk_lr, so its
// partial is bit-identical.  sqh / sql: the packed query rows, staged by
// the caller with attn_stage_q.  o[t]: rows 16 t + 4 g + i (i = 0..3), feature 16 wave + kl.
template <int CK, int T>
struct AttnSmemG {
  alignas(16) uint16_t ph[16 * T][CK + 8];
  alignas(16) uint16_t pl[16 * T][CK + 8];
  float pm[16 * T][8], ps[16 * T][8];
  float m[16 * T], l[16 * T];
};

// Query head within the group (gg) and request row (rw) of packed rows
// p0 + 16 t + i (t < T, i < NI), p0 + 16 t + i = gg R + rw: two divisions,
// then steps (a division per row costs some twenty VALU instructions).
template <int T, int NI>
__device__ __forceinline__ void attn_grp_rows(int p0, int R, int (&gg)[T][NI], int (&rw)[T][NI]) {
  const int sq = 16 / R, sr = 16 - sq * R;
  int q = p0 / R, r = p0 - q * R;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    int qi = q, ri = r;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      gg[t][i] = qi;
      rw[t][i] = ri;
      if (++ri == R) {
        ri = 0;
        ++qi;
      }
    }
    r += sr;
    q += sq;
    if (r >= R) {
      r -= R;
      ++q;
    }
  }
}

template <int CK, int T>
__device__ __forceinline__ void attn_chunk_grp(const AttnItem& it, const uint4 (&kf)[CK / 128][4],
                                               const uint16_t (*sqh)[kAttnQPitch],
                                               const uint16_t (*sql)[kAttnQPitch], int R, int NR, float scale,
                                               AttnSmemG<CK, T>& sm, floatx4 (&o)[T]) {
  constexpr int NG = CK / 128;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
  const int ke = (it.k_hi + 7) & ~7;
  int gg[T][4], rw[T][4];
  attn_grp_rows<T, 4>(4 * g, R, gg, rw);
  float sv[T][NG][4];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 qh = *(const uint4*)&sqh[16 * t + kl][32 * ks + 8 * g];
        const uint4 ql = *(const uint4*)&sql[16 * t + kl][32 * ks + 8 * g];
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ql),
                                                      __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qh),
                                                      __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
      }
      const int key = it.k_lo + (CK / 8) * wave + 16 * grp + kl;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int pr = 16 * t + 4 * g + i;
        sv[t][grp][i] = (pr < NR && key < it.k_hi && key <= it.L + rw[t][i]) ? acc[i] * scale : -INFINITY;
      }
    }
  __builtin_amdgcn_sched_barrier(0);
  AttnRegs<CK> r;
  const uint16_t* vfr = it.vc + v_cache_index(16 * wave + kl, it.k_lo + 8 * g, kAttnHd);
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const int kv0 = it.k_lo + 32 * ks + 8 * g;
    r.vf[ks] = make_uint4(0, 0, 0, 0);
    if (kv0 + 8 <= ke) r.vf[ks] = ld_stream_g128(vfr + ks * 512);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = sv[t][0][i];
#pragma unroll
      for (int grp = 1; grp < NG; ++grp) mx = fmaxf(mx, sv[t][grp][i]);
      mx = row16_max(mx);
      if (kl == 0) sm.pm[16 * t + 4 * g + i][wave] = mx;
    }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * t + 4 * g + i;
      const float4 a = *(const float4*)&sm.pm[row][0];
      const float4 b = *(const float4*)&sm.pm[row][4];
      const float M = fmaxf(fmaxf(fmaxf(a.x, a.y), fmaxf(a.z, a.w)), fmaxf(fmaxf(b.x, b.y), fmaxf(b.z, b.w)));
      float sum = 0.f;
#pragma unroll
      for (int grp = 0; grp < NG; ++grp) {
        const float e = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((sv[t][grp][i] - M) * 1.44269504088896341f);
        sum += e;
        const uint16_t h = f2bf_num(e);
        const int kc = (CK / 8) * wave + 16 * grp + kl;
        sm.ph[row][kc] = h;
        sm.pl[row][kc] = f2bf_num(e - bf2f(h));
      }
      sum = row16_sum(sum);
      if (kl == 0) sm.ps[row][wave] = sum;
    }
  __syncthreads();
  if (tid < NR) {
    float l = 0.f, M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      l += sm.ps[tid][w];
      M = fmaxf(M, sm.pm[tid][w]);
    }
    sm.m[tid] = M;
    sm.l[tid] = l;
  }
  attn_mask_tail(it, lane, r);
#pragma unroll
  for (int t = 0; t < T; ++t) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < CK / 32; ++ks) {
      const uint4 ph = *(const uint4*)&sm.ph[16 * t + kl][32 * ks + 8 * g];
      const uint4 pl = *(const uint4*)&sm.pl[16 * t + kl][32 * ks + 8 * g];
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pl),
                                                    __builtin_bit_cast(bf16x8, r.vf[ks]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ph),
                                                    __builtin_bit_cast(bf16x8, r.vf[ks]), acc, 0, 0, 0);
    }
    o[t] = acc;
  }
}

// Store the grouped chunk's partials where attn_publish stores each head's:
// packed row pr goes to query head kvh G + pr / R, row pr % R.
template <int CK, int T>
__device__ __forceinline__ void attn_publish_grp(const AttnItem& it, int kvh, int G, const floatx4 (&o)[T],
                                                 const AttnSmemG<CK, T>& sa, float* part_o, float* part_ml, int H,
                                                 int NC, int Rmax, int R) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
  const int NR = G * R;
  int gq[T][4], rw[T][4];
  attn_grp_rows<T, 4>(4 * g, R, gq, rw);
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int pr = 16 * t + 4 * g + i;
      if (pr < NR) {
        const size_t bh = (size_t)it.bl * H + kvh * G + gq[t][i];
        float* po = part_o + ((bh * NC + it.c) * Rmax + rw[t][i]) * kAttnHd + 16 * wave + kl;
        __hip_atomic_store(po, o[t][i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  if (tid < NR) {
    const int gg = tid / R, row = tid - gg * R;
    const size_t bh = (size_t)it.bl * H + kvh * G + gg;
    float* pml = part_ml + ((bh * NC + it.c) * Rmax + row) * 2;
    __hip_atomic_store(pml, sa.m[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(pml + 1, sa.l[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---------------------------------------------------------------------------
// Prefill attention: R prompt rows of a request (R > 16), appended at
// positions L .. L + R - 1, each attending causally to the cache and the
// rows before it.  The rows form 16-row tiles; tile t is computed as a verify
// call of its own (L + 16 t cached keys, up to 16 rows), operation for
// operation, so each row gets the verify path's result bit for bit: the same
// 256-key chunks, the same scores (the query's two bf16 terms against 16 keys
// per MFMA output tile, four 32-feature steps each), the same chunk softmax
// (row max and row sum over each 32-key slice, then over the eight slices in
// order), the same probabilities' two bf16 terms against V^T in 32-key steps,
// the same merge weights (attn_row_weights) and the same chunk-order sum
// (attn_acc1).  A row's result does not depend on which other rows share its
// tile: every product and reduction of a chunk is per row, and chunks past a
// row's position get weight zero.
//
// Where the verify kernel spreads one chunk over eight waves, here one wave
// runs a whole tile: the eight 32-key slices of a chunk one after another,
// with no barrier between them.  The W waves of a workgroup take W
// consecutive tiles of one (request, head) and share every K and V^T block:
// SK keys at a time, staged through a two-slot LDS ring (rows of 16-byte
// pieces XOR-swizzled by row, so the 16 rows a fragment read touches hit
// distinct banks), the next block's loads in flight while the current one is
// used.  Each chunk is walked twice: the first walk keeps every chunk's row
// max and row sum in LDS, the merge weights follow from them, and the second
// walk recomputes each chunk's probabilities, multiplies them with V and adds
// the result, times its weight, to the tile's running sums in registers.
// ---------------------------------------------------------------------------
template <int W, int SK>
struct AttnPfSmem {
  static_assert(SK == 64 || SK == 128, "staged blocks of 64 or 128 keys");
  uint4 st[2][SK * 16];                    // K: SK rows of 16 pieces; V^T: 128 rows of SK / 8 pieces
  uint16_t ph[W][16][40], pl[W][16][40];  // one 32-key step's probabilities, per wave (rows padded by 16 bytes)
};

// Dynamic LDS of the prefill attention: per wave, chunk and row a (max, sum)
// pair, then the merge weight in .x.
__host__ __device__ inline unsigned attn_prefill_dyn_bytes(int W, int NC) { return (unsigned)W * NC * 16 * 8; }

// piece c (8 features) of staged K row r; piece c (8 keys) of staged V^T row f
__device__ __forceinline__ int pf_k_at(int r, int c) { return r * 16 + (c ^ (r & 15)); }
// The K piece that staging thread e moves: row r (a position of the block),
// piece c, in the cache's fragment order (k_cache_index), so 64 consecutive
// threads read one 1 KB fragment: 16 positions x 32 features.
__device__ __forceinline__ void pf_k_piece(int e, int& r, int& c) {
  const int fr = e >> 6, ln = e & 63;
  r = 16 * (fr >> 2) + (ln & 15);
  c = 4 * (fr & 3) + (ln >> 4);
}
template <int SK>
__device__ __forceinline__ int pf_v_at(int f, int c) {
  constexpr int CPR = SK / 8;
  return f * CPR + (CPR == 16 ? (c ^ (f & 15)) : (c ^ ((f >> 1) & 7)));
}

// This thread's share of staged block b of chunk c: K (b < 256 / SK: keys
// c * 256 + b * SK ..) or V^T (keys c * 256 + (b - 256 / SK) * SK ..).  Keys
// at or past k_hi (V^T: 8-key pieces past ke) read as zero.
template <int W, int SK>
__device__ __forceinline__ void pf_fetch(int c, int b, int k_hi, int ke, const uint16_t* kc, const uint16_t* vc,
                                         uint4 (&r)[SK * 16 / (64 * W)]) {
  constexpr int PER = SK * 16 / (64 * W), NB = 256 / SK, CPR = SK / 8;
  const bool is_v = b >= NB;
  const int k0 = c * 256 + (is_v ? b - NB : b) * SK;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = (int)threadIdx.x + 64 * W * q;
    r[q] = make_uint4(0, 0, 0, 0);
    if (!is_v) {
      int row, pc;
      pf_k_piece(e, row, pc);
      if (k0 + row < k_hi) r[q] = *(const uint4*)(kc + k_cache_index(pc * 8, k0 + row, kAttnHd));
    } else {
      const int f = e / CPR, pc = e % CPR, key = k0 + 8 * pc;
      if (key + 8 <= ke) r[q] = *(const uint4*)(vc + v_cache_index(f, key, kAttnHd));
    }
  }
}

template <int W, int SK>
__device__ __forceinline__ void pf_stash(AttnPfSmem<W, SK>& s, int slot, int b, const uint4 (&r)[SK * 16 / (64 * W)]) {
  constexpr int PER = SK * 16 / (64 * W), NB = 256 / SK, CPR = SK / 8;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = (int)threadIdx.x + 64 * W * q;
    int kr, kpc;
    pf_k_piece(e, kr, kpc);
    s.st[slot][b < NB ? pf_k_at(kr, kpc) : pf_v_at<SK>(e / CPR, e % CPR)] = r[q];
  }
}

// Wave-local ordering of LDS traffic between the lanes of one wave.
__device__ __forceinline__ void pf_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// q: this request's query rows ([R][d], head h's features at h * kAttnHd);
// kc / vc: the K and V blocks of (request, K/V head); L: the request's
// cached keys; t0: the group's first tile (tile t0 + wave for this wave).
// out(row, dd, value) receives every output of the group's rows (row counted
// from the request's first prompt row).  mlw: W * NCP * 16 pairs; NCP bounds
// the chunks of any tile.  All 64 W threads call it.
template <int W, int SK, class Out>
__device__ __forceinline__ void attn_prefill_tiles(AttnPfSmem<W, SK>& s, float2* mlw, int NCP, const float* q,
                                                   int d, int h, const uint16_t* kc, const uint16_t* vc, int L,
                                                   int R, int t0, float scale, Out&& out) {
  constexpr int NB = 256 / SK, SPB = SK / 32, PER = SK * 16 / (64 * W);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, kl = lane & 15;
  const int ntile = (R + 15) / 16;
  const int tl = t0 + wave;                            // this wave's tile
  const int Rt = tl < ntile ? min(16, R - 16 * tl) : 0;  // its rows (0: idle)
  const int Lt = L + 16 * tl;
  const int nct = Rt > 0 ? (Lt + Rt + 255) / 256 : 0;
  // the group's furthest key: the end of its last tile
  const int tlast = min(t0 + W, ntile) - 1;
  const int kend = L + 16 * tlast + min(16, R - 16 * tlast);
  const int ncg = (kend + 255) / 256;
  float2* ml = mlw + (size_t)wave * NCP * 16;

  // this lane's query fragments (row kl of the tile, features 32 ks + 8 g ..),
  // as two bf16 terms; rows past the tile: zeros
  uint4 qh[4], ql[4];
  {
    const bool ok = kl < Rt;
    const float* qr = q + (size_t)(16 * tl + kl) * d + h * kAttnHd;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = 0.f;
      if (ok) {
        const float4 a = *(const float4*)(qr + 32 * ks + 8 * g), b = *(const float4*)(qr + 32 * ks + 8 * g + 4);
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
      }
      attn_split2(x, qh[ks], ql[ks]);
    }
  }

  // scores of staged K block b (slices b * SPB ..) of chunk c into sv
  auto scores = [&](const uint4* blk, int c, int b, float (&sv)[8][2][4]) {
    const int k_lo = c * 256, k_hi = min(k_lo + 256, Lt + Rt);
#pragma unroll
    for (int j = 0; j < SPB; ++j) {
      const int vw = b * SPB + j;  // the slice (the verify kernel's wave)
#pragma unroll
      for (int grp = 0; grp < 2; ++grp) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        const int r = 32 * j + 16 * grp + kl;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const uint4 kf = blk[pf_k_at(r, 4 * ks + g)];
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ql[ks]),
                                                        __builtin_bit_cast(bf16x8, kf), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qh[ks]),
                                                        __builtin_bit_cast(bf16x8, kf), acc, 0, 0, 0);
        }
        const int key = k_lo + 32 * vw + 16 * grp + kl;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          sv[vw][grp][i] = (key < k_hi && key <= Lt + 4 * g + i) ? acc[i] * scale : -INFINITY;
      }
    }
  };
  // chunk softmax of sv: probabilities in place, and each row's max and sum
  auto softmax = [&](float (&sv)[8][2][4], float (&m)[4], float (&l)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mw[8];
#pragma unroll
      for (int vw = 0; vw < 8; ++vw) mw[vw] = row16_max(fmaxf(sv[vw][0][i], sv[vw][1][i]));
      const float M = fmaxf(fmaxf(fmaxf(mw[0], mw[1]), fmaxf(mw[2], mw[3])), fmaxf(fmaxf(mw[4], mw[5]), fmaxf(mw[6], mw[7])));
      float lsum = 0.f, mm = -INFINITY;
#pragma unroll
      for (int vw = 0; vw < 8; ++vw) {
        float sum = 0.f;
#pragma unroll
        for (int grp = 0; grp < 2; ++grp) {
          const float e = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((sv[vw][grp][i] - M) * 1.44269504088896341f);
          sum += e;
          sv[vw][grp][i] = e;
        }
        lsum += row16_sum(sum);
        mm = fmaxf(mm, mw[vw]);
      }
      m[i] = mm;
      l[i] = lsum;
    }
  };

  uint4 pre[PER];
  // first walk: every chunk's row max and row sum
  pf_fetch<W, SK>(0, 0, kend, 0, kc, vc, pre);
  pf_stash(s, 0, 0, pre);
  __syncthreads();
  int slot = 0;
  for (int c = 0; c < ncg; ++c) {
    float sv[8][2][4];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bool more = b + 1 < NB || c + 1 < ncg;
      if (more) pf_fetch<W, SK>(b + 1 < NB ? c : c + 1, b + 1 < NB ? b + 1 : 0, kend, 0, kc, vc, pre);
      if (c < nct) scores(s.st[slot], c, b, sv);
      if (more) pf_stash(s, slot ^ 1, 0, pre);
      __syncthreads();
      slot ^= 1;
    }
    if (c < nct) {
      float m[4], l[4];
      softmax(sv, m, l);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (kl == 0 && 4 * g + i < Rt) ml[c * 16 + 4 * g + i] = make_float2(m[i], l[i]);
    }
  }
  // merge weights of this wave's rows, in place of (max, sum)
  pf_wave_sync();
  for (int row = 0; row < Rt; ++row)
    attn_row_weights(
        nct,
        [&](int c, bool ok, float& m, float& l) {
          const float2 v = ok ? ml[c * 16 + row] : make_float2(0.f, 0.f);
          m = v.x;
          l = v.y;
        },
        [&](int c, float w) { ml[c * 16 + row].x = w; });
  pf_wave_sync();

  // second walk: K blocks (scores, softmax), then V^T blocks (P V), per chunk
  const int keg = (kend + 7) & ~7;
  float O[8][4];
#pragma unroll
  for (int fb = 0; fb < 8; ++fb)
#pragma unroll
    for (int i = 0; i < 4; ++i) O[fb][i] = 0.f;
  pf_fetch<W, SK>(0, 0, kend, keg, kc, vc, pre);
  pf_stash(s, slot, 0, pre);
  __syncthreads();
  for (int c = 0; c < ncg; ++c) {
    const int k_lo = c * 256, k_hi = min(k_lo + 256, Lt + Rt);
    float sv[8][2][4];
    floatx4 o[8];
#pragma unroll
    for (int fb = 0; fb < 8; ++fb) o[fb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < 2 * NB; ++b) {
      const bool more = b + 1 < 2 * NB || c + 1 < ncg;
      if (more) pf_fetch<W, SK>(b + 1 < 2 * NB ? c : c + 1, b + 1 < 2 * NB ? b + 1 : 0, kend, keg, kc, vc, pre);
      if (c < nct) {
        if (b < NB) {
          scores(s.st[slot], c, b, sv);
          if (b == NB - 1) {
            float m[4], l[4];
            softmax(sv, m, l);
          }
        } else {
          const uint4* blk = s.st[slot];
#pragma unroll
          for (int j = 0; j < SPB; ++j) {
            const int ks = (b - NB) * SPB + j;  // 32-key step of the chunk
            // this step's probabilities, as two bf16 terms, through LDS into
            // the A-operand layout (row kl, keys 8 g ..)
#pragma unroll
            for (int grp = 0; grp < 2; ++grp)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const float e = sv[ks][grp][i];
                const uint16_t hb = f2bf_num(e);
                s.ph[wave][4 * g + i][16 * grp + kl] = hb;
                s.pl[wave][4 * g + i][16 * grp + kl] = f2bf_num(e - bf2f(hb));
              }
            pf_wave_sync();
            const uint4 pa_h = *(const uint4*)&s.ph[wave][kl][8 * g];
            const uint4 pa_l = *(const uint4*)&s.pl[wave][kl][8 * g];
            const int kv0 = k_lo + 32 * ks + 8 * g;
#pragma unroll
            for (int fb = 0; fb < 8; ++fb) {
              uint4 vf = blk[pf_v_at<SK>(16 * fb + kl, 4 * j + g)];
              if (kv0 + 8 > k_hi) {  // this tile's keys only (the verify kernel's tail mask)
                uint32_t wv[4] = {vf.x, vf.y, vf.z, vf.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const int p0 = kv0 + 2 * e;
                  if (p0 >= k_hi) wv[e] = 0u;
                  else if (p0 + 1 >= k_hi) wv[e] &= 0xffffu;
                }
                vf = make_uint4(wv[0], wv[1], wv[2], wv[3]);
              }
              o[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pa_l),
                                                              __builtin_bit_cast(bf16x8, vf), o[fb], 0, 0, 0);
              o[fb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pa_h),
                                                              __builtin_bit_cast(bf16x8, vf), o[fb], 0, 0, 0);
            }
            pf_wave_sync();
          }
        }
      }
      if (more) pf_stash(s, slot ^ 1, b + 1 < 2 * NB ? b + 1 : 0, pre);
      __syncthreads();
      slot ^= 1;
    }
    if (c < nct) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * g + i;
        const float w = row < Rt ? ml[c * 16 + row].x : 0.f;
#pragma unroll
        for (int fb = 0; fb < 8; ++fb) O[fb][i] = attn_acc1(O[fb][i], o[fb][i], w);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * g + i;
    if (row < Rt)
#pragma unroll
      for (int fb = 0; fb < 8; ++fb) out(16 * tl + row, 16 * fb + kl, O[fb][i]);
  }
}

}  // namespace spade
