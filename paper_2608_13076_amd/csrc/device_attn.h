// Verify attention for a bf16 cache with head_dim 128 (Sec. III-A: the
// gamma+1 appended rows of a request attend causally to its cached keys and
// to each other), shared by the per-stage kernels and the persistent verify
// kernel.
//
// Work item: (request, head, chunk of kAttnChunkB keys), one 8-wave
// workgroup; wave w owns keys [k_lo + 32 S w, k_lo + 32 S (w + 1)) as S =
// kAttnSub sub-blocks of 32 keys.  Row i of the request sits at position L + i and sees keys
// <= L + i.  Scores S = Q K^T and O = P V run on MFMA 16x16x32 bf16 with Q and
// P split into two bf16 terms (hi + lo); K is stored as rows [pos][hd] and V
// transposed, rows [feature][stride], so both B operands are 16-byte loads.
// A chunk writes its unnormalised output, row max and row sum; the chunks of
// a (request, head) are merged in chunk order with weights
// exp(m_c - max) / sum_c(l_c exp(m_c - max)) (attn_merge_weights).
#pragma once

#include "device_util.h"

namespace spade {

constexpr int kAttnSub = 1;                    // 32-key sub-blocks per wave
constexpr int kAttnChunkB = 8 * 32 * kAttnSub;  // keys per chunk (8 waves)
constexpr int kAttnHd = 128;
constexpr int kAttnRows = 16;      // rows per request (gamma + 1 <= 16)

struct AttnSmemB {
  float s[kAttnRows][kAttnChunkB];  // scores, then probabilities
  float o[8][kAttnRows][kAttnHd];   // per-wave partial outputs
  float m[kAttnRows], l[kAttnRows];
};

struct AttnRegsB {
  uint4 kf[kAttnSub][2][4];  // [sub-block][16-key group][32-feature slice]
  uint4 vf[kAttnSub][8];     // [sub-block][16-feature tile]: this lane's 8 keys
};

struct AttnItemB {
  bool active;
  int bl, h, c;
  int L;           // cached keys of the request (row i sits at L + i)
  int k_lo, k_hi;  // keys of this chunk: [k_lo, k_hi)
  const uint16_t* kc;  // K rows of (request, head)
  const uint16_t* vc;  // V^T rows of (request, head)
};

__device__ __forceinline__ void attn_zero_regs(AttnRegsB& r) {
#pragma unroll
  for (int sb = 0; sb < kAttnSub; ++sb) {
#pragma unroll
    for (int grp = 0; grp < 2; ++grp)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) r.kf[sb][grp][ks] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int ft = 0; ft < 8; ++ft) r.vf[sb][ft] = make_uint4(0, 0, 0, 0);
  }
}

// Keys of this wave in [kb, ke) (plain loads).  V^T vectors load whole when
// all their 8 keys are in [kb, ke); keys at or past k_hi read as zero.
__device__ __forceinline__ void attn_load_plain(const AttnItemB& it, int stride, int kb, int ke, int wave, int lane,
                                                AttnRegsB& r) {
  const int g = lane >> 4, kl = lane & 15;
#pragma unroll
  for (int sb = 0; sb < kAttnSub; ++sb) {
    const int kw = it.k_lo + 32 * kAttnSub * wave + 32 * sb;
#pragma unroll
    for (int grp = 0; grp < 2; ++grp) {
      const int key = kw + 16 * grp + kl;
      if (key >= kb && key < ke && key < it.k_hi) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) r.kf[sb][grp][ks] = *(const uint4*)(it.kc + (size_t)key * kAttnHd + 32 * ks + 8 * g);
      }
    }
    const int kv0 = kw + 8 * g;
    if (kv0 >= kb && kv0 + 8 <= ke) {
#pragma unroll
      for (int ft = 0; ft < 8; ++ft) r.vf[sb][ft] = *(const uint4*)(it.vc + (size_t)(16 * ft + kl) * stride + kv0);
    }
  }
}

// The keys this verify call appended, [L, k_hi), written earlier in the same
// launch by other workgroups: sc1 loads (rk, rv: resources over this (request,
// head)'s K and V^T rows).  A V^T vector holding any such key loads whole.
__device__ __forceinline__ void attn_load_new(const AttnItemB& it, Rsrc rk, Rsrc rv, int stride, int wave, int lane,
                                              AttnRegsB& r) {
  const int g = lane >> 4, kl = lane & 15;
#pragma unroll
  for (int sb = 0; sb < kAttnSub; ++sb) {
    const int kw = it.k_lo + 32 * kAttnSub * wave + 32 * sb;
#pragma unroll
    for (int grp = 0; grp < 2; ++grp) {
      const int key = kw + 16 * grp + kl;
      if (key >= it.L && key < it.k_hi) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
          r.kf[sb][grp][ks] = ld_b128<true>(rk, (uint32_t)(key * kAttnHd + 32 * ks + 8 * g) * 2u);
      }
    }
    const int kv0 = kw + 8 * g;
    if (kv0 + 8 > it.L && kv0 < it.k_hi) {
#pragma unroll
      for (int ft = 0; ft < 8; ++ft) r.vf[sb][ft] = ld_b128<true>(rv, (uint32_t)((16 * ft + kl) * stride + kv0) * 2u);
    }
  }
}

// Zero the V^T entries of keys at or past k_hi (their P is zero, but the
// cache may hold anything there).
__device__ __forceinline__ void attn_mask_tail(const AttnItemB& it, int wave, int lane, AttnRegsB& r) {
  const int g = lane >> 4;
#pragma unroll
  for (int sb = 0; sb < kAttnSub; ++sb) {
    const int kv0 = it.k_lo + 32 * kAttnSub * wave + 32 * sb + 8 * g;
    if (kv0 + 8 > it.k_hi) {
#pragma unroll
      for (int ft = 0; ft < 8; ++ft) {
        uint32_t w[4] = {r.vf[sb][ft].x, r.vf[sb][ft].y, r.vf[sb][ft].z, r.vf[sb][ft].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int p0 = kv0 + 2 * e;
          if (p0 >= it.k_hi) w[e] = 0u;
          else if (p0 + 1 >= it.k_hi) w[e] &= 0xffffu;
        }
        r.vf[sb][ft] = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
  }
}

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

// One chunk with K/V fragments in r.  q: row 0 of the request's rotated
// queries for this head (rows R apart by q_stride floats).  On return
// sm.o[0..7] hold the wave partials, sm.m / sm.l the row max / sum (for an
// empty chunk -inf / 0).  All 512 threads call it (it synchronises).
__device__ __forceinline__ void attn_chunk(const AttnItemB& it, const float* q, int q_stride, int R, float scale,
                                           AttnRegsB& r, AttnSmemB& sm) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, kl = lane & 15;
  uint4 qh[4], ql[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    qh[ks] = make_uint4(0, 0, 0, 0);
    ql[ks] = make_uint4(0, 0, 0, 0);
  }
  if (it.active && kl < R) {
    const float* qp = q + (size_t)kl * q_stride + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float4 x0 = *(const float4*)(qp + 32 * ks);
      const float4 x1 = *(const float4*)(qp + 32 * ks + 4);
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      attn_split2(xs, qh[ks], ql[ks]);
    }
  }
  // S = Q K^T; D[i][j] sits in lane j + 16*(i/4), register i%4: rows 4g..4g+3 of key kl
#pragma unroll
  for (int sb = 0; sb < kAttnSub; ++sb)
#pragma unroll
    for (int grp = 0; grp < 2; ++grp) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ql[ks]),
                                                      __builtin_bit_cast(bf16x8, r.kf[sb][grp][ks]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qh[ks]),
                                                      __builtin_bit_cast(bf16x8, r.kf[sb][grp][ks]), acc, 0, 0, 0);
      }
      const int key = it.k_lo + 32 * kAttnSub * wave + 32 * sb + 16 * grp + kl;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * g + i;
        if (key < it.k_hi) sm.s[row][key - it.k_lo] = (key <= it.L + row) ? acc[i] * scale : -INFINITY;
      }
    }
  __syncthreads();
  // chunk softmax, one wave per row; keys past the chunk end get p = 0
  const int nk = it.k_hi - it.k_lo;
  for (int row = wave; row < R; row += 8) {
    float mx = -INFINITY;
    for (int j = lane; j < nk; j += 64) mx = fmaxf(mx, sm.s[row][j]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    float sum = 0.f;
    for (int j = lane; j < kAttnChunkB; j += 64) {
      const float e = (j < nk && mx != -INFINITY) ? expf(sm.s[row][j] - mx) : 0.f;
      sm.s[row][j] = e;
      sum += e;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
    if (lane == 0) {
      sm.m[row] = mx;
      sm.l[row] = sum;
    }
  }
  __syncthreads();
  // O = P V over the wave's keys (sub-blocks in order)
  floatx4 oacc[8];
#pragma unroll
  for (int ft = 0; ft < 8; ++ft) oacc[ft] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int sb = 0; sb < kAttnSub; ++sb) {
    uint4 ph = make_uint4(0, 0, 0, 0), pl = make_uint4(0, 0, 0, 0);
    if (kl < R) {
      const float* pp = &sm.s[kl][32 * kAttnSub * wave + 32 * sb + 8 * g];
      const float4 x0 = *(const float4*)pp;
      const float4 x1 = *(const float4*)(pp + 4);
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      attn_split2(xs, ph, pl);
    }
#pragma unroll
    for (int ft = 0; ft < 8; ++ft) {
      oacc[ft] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pl),
                                                         __builtin_bit_cast(bf16x8, r.vf[sb][ft]), oacc[ft], 0, 0, 0);
      oacc[ft] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ph),
                                                         __builtin_bit_cast(bf16x8, r.vf[sb][ft]), oacc[ft], 0, 0, 0);
    }
  }
#pragma unroll
  for (int ft = 0; ft < 8; ++ft)
#pragma unroll
    for (int i = 0; i < 4; ++i) sm.o[wave][4 * g + i][16 * ft + kl] = oacc[ft][i];
  __syncthreads();
}

// Unnormalised chunk output of (row, dd): the eight wave partials in order.
__device__ __forceinline__ float attn_chunk_out(const AttnSmemB& sm, int row, int dd) {
  float v = sm.o[0][row][dd];
#pragma unroll
  for (int w = 1; w < 8; ++w) v += sm.o[w][row][dd];
  return v;
}

// Merge weights of row `row` from (m, l) pairs ml[2 * (c * R + row)]: the
// weight of chunk c is exp(m_c - max) / sum_c(l_c exp(m_c - max)), written to
// sc[c * R + row].
__device__ __forceinline__ void attn_merge_weights(const float* ml, float* sc, int NC, int R, int row) {
  float Mx = -INFINITY;
  for (int c = 0; c < NC; ++c) Mx = fmaxf(Mx, ml[2 * (c * R + row)]);
  float Ls = 0.f;
  for (int c = 0; c < NC; ++c) {
    const float mc = ml[2 * (c * R + row)];
    const float e = (mc == -INFINITY) ? 0.f : expf(mc - Mx);
    Ls += ml[2 * (c * R + row) + 1] * e;
    sc[c * R + row] = e;
  }
  const float inv = 1.0f / Ls;
  for (int c = 0; c < NC; ++c) sc[c * R + row] *= inv;
}

// Last-arrival merge of the chunks of one (request, head).
struct AttnMergeSmem {
  float ml[2 * kAttnMaxChunks * kAttnRows];  // (m, l) of every chunk, [c][row][2]
  float sc[kAttnMaxChunks * kAttnRows];      // merge weights, [c][row]
  int last;
};

// partials of output o (= row * kAttnHd + dd) for chunks 0..7 (sc1 loads)
__device__ __forceinline__ void attn_load8(Rsrc rpo, int NC, int Rmax, int o, bool ok, float (&v)[8]) {
  const int row = o / kAttnHd, dd = o - row * kAttnHd;
#pragma unroll
  for (int c = 0; c < 8; ++c)
    v[c] = ld_b32_coh(rpo, (ok && c < NC) ? (uint32_t)((c * Rmax + row) * kAttnHd + dd) * 4u : kOob);
}

// weighted sum of output o over the chunks, in chunk order
__device__ __forceinline__ float attn_merged(Rsrc rpo, const AttnMergeSmem& ms, int NC, int Rmax, int R, int o,
                                             const float (&v)[8]) {
  const int row = o / kAttnHd, dd = o - row * kAttnHd;
  float O = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    if (c < NC) {
      const float w = ms.sc[c * R + row];
      O += w != 0.f ? v[c] * w : 0.f;
    }
  }
  for (int c = 8; c < NC; ++c) {
    const float w = ms.sc[c * R + row];
    const float val = ld_b32_coh(rpo, (uint32_t)((c * Rmax + row) * kAttnHd + dd) * 4u);
    O += w != 0.f ? val * w : 0.f;
  }
  return O;
}

// Publish this chunk's partial with write-through stores, arrive on the
// counter of its (request, head) once the stores have landed, and, in the
// workgroup that arrives last, merge all chunks in chunk order (weights
// attn_merge_weights) and pass each merged output o = row * kAttnHd + dd to
// out(o, value).  The last arrival resets the counter.  part_o / part_ml:
// [bh][NC][Rmax][kAttnHd] / [bh][NC][Rmax][2].  All 512 threads call it.
template <class Out>
__device__ __forceinline__ void attn_publish_merge(const AttnItemB& it, const AttnSmemB& sa, AttnMergeSmem& ms,
                                                   float* part_o, float* part_ml, uint32_t* attn_cnt, int H,
                                                   int NC, int Rmax, int R, Out&& out) {
  const int tid = threadIdx.x;
  const size_t bh = (size_t)it.bl * H + it.h;
  if (it.active) {
    float* po = part_o + ((bh * NC + it.c) * Rmax) * kAttnHd;
    float* pml = part_ml + ((bh * NC + it.c) * Rmax) * 2;
    for (int idx = tid; idx < R * kAttnHd; idx += 512) {
      const int row = idx / kAttnHd, dd = idx - row * kAttnHd;
      __hip_atomic_store(po + row * kAttnHd + dd, attn_chunk_out(sa, row, dd), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tid < R) {
      __hip_atomic_store(pml + tid * 2, sa.m[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(pml + tid * 2 + 1, sa.l[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) {
    int last = 0;
    if (it.active) {
      uint32_t* cnt = attn_cnt + bh;
      const uint32_t o = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (o == (uint32_t)NC - 1u) {
        __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = 1;
      }
    }
    ms.last = last;
  }
  __syncthreads();
  if (!ms.last) return;  // uniform across the workgroup
  // the (m, l) pairs and this thread's first partials in one round trip
  const Rsrc rpo = wave_rsrc(part_o + (bh * NC * Rmax) * kAttnHd);
  const Rsrc rpm = wave_rsrc(part_ml + (bh * NC * Rmax) * 2);
  const int nout = R * kAttnHd;
  float v0[8], v1[8];
  attn_load8(rpo, NC, Rmax, tid, tid < nout, v0);
  attn_load8(rpo, NC, Rmax, tid + 512, tid + 512 < nout, v1);
  for (int i = tid; i < NC * R; i += 512) {
    const int c = i / R, row = i - c * R;
    const uint32_t off = (uint32_t)((c * Rmax + row) * 2) * 4u;
    ms.ml[2 * i] = ld_b32_coh(rpm, off);
    ms.ml[2 * i + 1] = ld_b32_coh(rpm, off + 4u);
  }
  __syncthreads();
  if (tid < R) attn_merge_weights(ms.ml, ms.sc, NC, R, tid);
  __syncthreads();
  if (tid < nout) out(tid, attn_merged(rpo, ms, NC, Rmax, R, tid, v0));
  if (tid + 512 < nout) out(tid + 512, attn_merged(rpo, ms, NC, Rmax, R, tid + 512, v1));
  for (int o = tid + 1024; o < nout; o += 512) {
    float v[8];
    attn_load8(rpo, NC, Rmax, o, true, v);
    out(o, attn_merged(rpo, ms, NC, Rmax, R, o, v));
  }
}

}  // namespace spade
