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
// MFMA 16x16x32 bf16 with Q and P split into two bf16 terms (hi + lo).  K is
// stored as rows [pos][hd] and V transposed, rows [feature][stride], so both
// B operands are 16-byte loads.  A chunk writes its unnormalised output, row
// max and row sum; the chunks of a (request, head) are merged in chunk order
// with weights exp(m_c - max) / sum_c(l_c exp(m_c - max)).
#pragma once

#include "device_util.h"

namespace spade {

constexpr int kAttnHd = 128;
constexpr int kAttnRows = 16;  // rows per request (gamma + 1 <= 16)
constexpr int kAttnThreads = 512;

template <int CK>
struct AttnSmem {
  static_assert(CK == 128 || CK == 256, "chunk of 128 or 256 keys");
  // probabilities as two bf16 terms (the A operand of O = P V); rows padded by
  // 16 bytes so the 16 rows of a fragment read start in different banks
  uint16_t ph[kAttnRows][CK + 8], pl[kAttnRows][CK + 8];
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
  const uint16_t* kc;  // K rows of (request, head)
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
      for (int ks = 0; ks < 4; ++ks) kf[grp][ks] = *(const uint4*)(it.kc + (size_t)key * kAttnHd + 32 * ks + 8 * g);
    }
  }
}

template <int CK>
__device__ __forceinline__ floatx4 attn_chunk_lr(const AttnItem& it, const uint4 (&kf)[CK / 128][4],
                                                 const uint16_t (*sqh)[kAttnQPitch],
                                                 const uint16_t (*sql)[kAttnQPitch], int R, float scale, int stride,
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
  // the V^T fragments, after the score products (the K registers are free)
  __builtin_amdgcn_sched_barrier(0);
  AttnRegs<CK> r;
  const uint16_t* vrow = it.vc + (size_t)(16 * wave + kl) * stride;
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const int kv0 = it.k_lo + 32 * ks + 8 * g;
    r.vf[ks] = make_uint4(0, 0, 0, 0);
    if (kv0 + 8 <= ke) r.vf[ks] = *(const uint4*)(vrow + kv0);
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

// add chunks c0 .. c0 + 15 of output o to O, in chunk order
__device__ __forceinline__ void attn_acc16(const AttnMergeSmem& ms, int c0, int nc, int o, const float (&v)[16],
                                           float& O) {
  const int row = o / kAttnHd;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int c = c0 + j;
    if (c < nc) {
      const float w = ms.sc[c][row];
      O += w != 0.f ? v[j] * w : 0.f;
    }
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
  constexpr int NJ = kAttnMaxChunks / 64;
  float mc[2][NJ], lc[2][NJ];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int row = wave + 8 * k;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = lane + 64 * j;
      const bool ok = row < R && c < nc;
      const uint32_t off = ok ? (uint32_t)((c * Rmax + row) * 2) * 4u : kOob;
      const float m = ld_f32<COH>(rpm, off);
      mc[k][j] = ok ? m : -INFINITY;
      lc[k][j] = ld_f32<COH>(rpm, off == kOob ? kOob : off + 4u);
    }
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int row = wave + 8 * k;
    if (row < R) {  // uniform across the wave
      float Mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < NJ; ++j) Mx = fmaxf(Mx, mc[k][j]);
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) Mx = fmaxf(Mx, __shfl_xor(Mx, off));
      float Ls = 0.f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        mc[k][j] = (mc[k][j] == -INFINITY) ? 0.f : expf(mc[k][j] - Mx);
        Ls += lc[k][j] * mc[k][j];
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) Ls += __shfl_xor(Ls, off);
      const float inv = 1.0f / Ls;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int c = lane + 64 * j;
        if (c < nc) ms.sc[c][row] = mc[k][j] * inv;
      }
    }
  }
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
  uint16_t ph[16 * T][CK + 8], pl[16 * T][CK + 8];
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
                                               int stride, AttnSmemG<CK, T>& sm, floatx4 (&o)[T]) {
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
  const uint16_t* vrow = it.vc + (size_t)(16 * wave + kl) * stride;
#pragma unroll
  for (int ks = 0; ks < CK / 32; ++ks) {
    const int kv0 = it.k_lo + 32 * ks + 8 * g;
    r.vf[ks] = make_uint4(0, 0, 0, 0);
    if (kv0 + 8 <= ke) r.vf[ks] = *(const uint4*)(vrow + kv0);
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

}  // namespace spade
