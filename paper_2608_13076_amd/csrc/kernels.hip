// HIP kernels of the speculative-verify path for gfx950 (MI355X).
//
// One verify pass of SPADE's cloud verifier (Algorithm 1, Cloud step): the
// gamma+1 rows [pending, d_1 .. d_gamma] of every request go through the
// decoder in one pass (Sec. III-A), the LM-head logits give the softmax rows,
// and the accept/reject chain with its correction draw (Sec. III-C) runs on
// the device.
//
// Kernels
//   embed_kernel   x = E[token]; first GEMM operand and RMS partials
//   gemm_kernel    Y = X W^T for skinny X (<= 32 rows) against bf16 or f32
//                  weights streamed from a tiled arena by persistent
//                  workgroups, double-buffered; MFMA 16x16x32 bf16 (fp32
//                  activations split into two bf16 terms) or 16x16x4 f32;
//                  fused epilogues: RMSNorm scale + RoPE + KV append (QKV),
//                  residual add + next RMS partials (O, down), SiLU gate
//                  (gate/up), logits + per-panel softmax statistics (LM head)
//   gemm_split_kernel  the same with the k-blocks of each panel split over
//                  2 or 4 workgroups (few panels, long K: the down projection)
//   gemm_wide_kernel   the same epilogues for more than 16 rows: row tiles
//                  and panels per workgroup, the operand through an LDS ring,
//                  optional k-splits for the O and down projections
//   gemm_mid_kernel    batched-verification projections of up to 144 rows:
//                  every row x 256 columns per workgroup, k-split, sums
//                  published; gemm_mid_finish_kernel adds them in range
//                  order and runs the epilogue
//   gemm_big_kernel    the projections of prefill forwards (hundreds to
//                  thousands of rows): 128 rows x 256 columns per workgroup
//   attn_lr_kernel the bf16 / head_dim-128 verify attention, one 256-key
//                  chunk per workgroup; merges the chunks of a (request,
//                  head) in the last one to finish, or leaves that to
//   attn_merge_kernel  a second launch (several rounds of chunk workgroups)
//   attn_g_kernel  grouped-query models: a chunk for all query heads of a
//                  K/V head in one workgroup (merged by attn_merge_kernel)
//   attn_kernel / attn_combine_kernel  f32 cache or other head sizes:
//                  128-key chunks, then the chunk-order merge
//   attn_prefill_kernel  prefill forwards of more than 16 rows per request:
//                  one wave per 16-row tile, each tile computed as a verify
//                  call of its own, K / V^T blocks shared through LDS
//   accept_kernel  per request: vocabulary-wide max / log-sum-exp / argmax
//                  per row, the accept chain, the Gumbel-max correction draw
//   correct_kernel that draw over vocabulary slices (calls that may sample)
//   commit_kernel  lens += n + 1, pending = correction
//   copy_state_kernel / advance_kernel  cache-state copies and single-request
//                  prefill bookkeeping
//   prefill_*_kernel   batched prefill: counts and start lengths, token
//                  gather, advance, pending
//   softmax_rows_kernel  softmax of logits / T (the draft side of Algorithm 1)
//   pack_kernel    row-major weights -> tiled arena
#include "device_accept.h"
#include "device_attn.h"
#include "device_gemm.h"
#include "device_gemm_big.h"
#include "device_gemm_mid.h"
#include "device_gemm_split.h"
#include "device_gemm_wide.h"

#include <float.h>
#include <math.h>

#include <algorithm>
#include <mutex>

namespace spade {

// Store v as the next GEMM's operand: kActSplits bf16 terms (bf16 weights:
// hi = rne(v), lo = rne(v - hi)) or the float itself (fp32 weights).
template <bool ABF16>
__device__ __forceinline__ void store_act(void* base, size_t split, size_t idx, float v) {
  if constexpr (ABF16) {
    uint16_t* p = (uint16_t*)base;
    float r = v;
#pragma unroll
    for (int s = 0; s < kActSplits; ++s) {
      const uint16_t h = f2bf(r);
      p[s * split + idx] = h;
      r -= bf2f(h);
    }
  } else {
    ((float*)base)[idx] = v;
  }
}

// ---------------------------------------------------------------------------
// Embedding: x_0 = E[token] (Sec. III-A), written with the split operand of
// the first QKV GEMM (x * g_attn of layer 0) and per-16-column sums of x^2.
// ---------------------------------------------------------------------------
struct EmbedParams {
  const void* E;
  const float* g;
  const int32_t* tokens;   // prefill ids [nb][R] or NULL
  const int32_t* drafts;   // [nb][R-1]
  const int32_t* pending;  // global [Bmax]
  int b0, R, d, V;
  float* x;
  void* act;
  size_t act_split;
  float* ssq;
  uint32_t* err;
  int32_t* lens;   // global [Bmax] cached lengths
  int len_limit;   // lens[b] + R may not exceed this (cache capacity, attention coverage)
};

template <bool WBF16>
__global__ void __launch_bounds__(256) embed_kernel(EmbedParams p) {
  const int m = blockIdx.x;
  const int bl = m / p.R, i = m % p.R;
  // A length the host could not bound (lens written outside the library's
  // calls): clamp it so every later kernel of the call stays inside the cache
  // and the attention's chunk grid, and flag the call.  The later kernels run
  // after this one on the same stream.
  if (i == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
    const int L = p.lens[p.b0 + bl];
    if (L < 0 || L > p.len_limit - p.R) {
      flag_error(p.err, SPADE_DERR_CAPACITY);
      p.lens[p.b0 + bl] = L < 0 ? 0 : p.len_limit - p.R;
    }
  }
  int t;
  if (p.tokens) t = p.tokens[m];
  else t = (i == 0) ? p.pending[p.b0 + bl] : p.drafts[bl * (p.R - 1) + i - 1];
  if (t < 0 || t >= p.V) {
    if (threadIdx.x == 0 && blockIdx.y == 0) flag_error(p.err, SPADE_DERR_TOKEN);
    t = t < 0 ? 0 : p.V - 1;
  }
  // one column per thread; the sixteen lanes of a panel sum x^2 in a fixed
  // butterfly order
  const int npan = p.d / 16;
  for (int n0 = (int)(blockIdx.y * blockDim.x); n0 < p.d; n0 += (int)(blockDim.x * gridDim.y)) {
    const int n = n0 + (int)threadIdx.x;
    const bool ok = n < p.d;
    float v = 0.f;
    if (ok) {
      if constexpr (WBF16) v = bf2f(((const uint16_t*)p.E)[(size_t)t * p.d + n]);
      else v = ((const float*)p.E)[(size_t)t * p.d + n];
      p.x[(size_t)m * p.d + n] = v;
      store_act<WBF16>(p.act, p.act_split, (size_t)m * p.d + n, v * p.g[n]);
    }
    float ss = v * v;
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    if (ok && (n & 15) == 0) p.ssq[(size_t)m * npan + (n >> 4)] = ss;
  }
}

// ---------------------------------------------------------------------------
// Projection GEMMs (engine in device_gemm.h): one launch per (layer, kind,
// block of <= 32 rows), persistent workgroups.
// ---------------------------------------------------------------------------
template <bool WBF16, int MT, bool ALDS, int KIND>
__global__ void __launch_bounds__(kGemmWaves * 64) gemm_kernel(GemmParams a) {
  __shared__ GemmSmem<MT> sm;
  extern __shared__ uint4 lds_dyn[];
  Gemm<WBF16, MT, ALDS, KIND, false> g(a, sm, (uint8_t*)lds_dyn, (int)blockIdx.x, (int)gridDim.x);
  g.run();
}

// Split-K skinny projection GEMM (device_gemm_split.h): G workgroups per
// k-split, workgroup b in split b / G.
constexpr uint32_t kSplitSmemBytes = (uint32_t)((sizeof(GemmSplitSmem) + 15) / 16 * 16);

template <int KS, int KIND>
__global__ void __launch_bounds__(kGemmWaves * 64) gemm_split_kernel(GemmParams a, uint32_t* cnt, float* part, int G) {
  extern __shared__ uint4 lds_dyn[];
  GemmSplit<KS, KIND> g(a, *(GemmSplitSmem*)lds_dyn, (uint8_t*)lds_dyn + kSplitSmemBytes, cnt, part, G);
  g.run();
}

// Wide-row projection GEMM (device_gemm_wide.h): workgroup b runs on XCD
// b % 8 and takes unit group b % 8 + 8 (q / (NRG KS)), then k-split and row
// group from q % (NRG KS) (row group fastest), q = b / 8, so the row groups
// and k-splits of a unit group share that XCD's L2.  K-splits: cnt / part
// hold one arrival counter / kWideItemFloats published values per (unit
// group, row group).
// Large-M projections (device_gemm_big.h): workgroup (row group, panel
// group).  Workgroup b runs on XCD b % 8, which owns panel groups b % 8 + 8 c;
// its workgroups go in blocks of 4 row groups x every one of its panel
// groups, so the workgroups that run together on an XCD share both their
// weight panels and their activation rows in its L2.
template <int KIND>
__global__ void __launch_bounds__(kBigWaves * 64)
gemm_big_kernel(GemmParams a, int NRG, int NUG) {
  extern __shared__ uint4 lds_dyn[];
  const int b = (int)blockIdx.x, q = b >> 3;
  const int NC = (NUG + 7) / 8;     // panel groups per XCD
  constexpr int RB = 4;             // row groups per block
  const int full = NRG / RB;        // whole blocks
  int rg, c;
  if (q < full * RB * NC) {
    const int blk = q / (RB * NC), w = q - blk * (RB * NC);
    c = w / RB;
    rg = blk * RB + (w - c * RB);
  } else {
    const int rbs = NRG - full * RB, w = q - full * RB * NC;  // the last, partial block
    c = w / rbs;
    rg = full * RB + (w - c * rbs);
  }
  const int ug = (b & 7) + 8 * c;
  if (ug >= NUG) return;  // uniform, before any barrier
  GemmBig<KIND> gb(a, *(GemmBigSmem*)lds_dyn, rg, ug);
  gb.run();
}

// Batched-verification projections of up to 144 rows
// (device_gemm_mid.h), first pass: workgroup b = (panel group b / KS, k-split
// b % KS) publishes its sums into part (kMidItemFloats per panel group).
template <int KIND>
__global__ void __launch_bounds__(kMidWaves * 64)
gemm_mid_kernel(GemmParams a, int NUG, int KS, float* part) {
  extern __shared__ uint4 lds_dyn[];
  const int b = (int)blockIdx.x;
  const int ug = b / KS, ks = b - ug * KS;
  if (ug >= NUG) return;  // uniform, before any barrier
  GemmMid<KIND> g(a, *(GemmMidSmem*)lds_dyn, ug, ks, KS, part + (size_t)ug * kMidItemFloats);
  g.run();
}

// Second pass: workgroup b = (panel group b / kMidRT, row tile b % kMidRT)
// adds the published sums in range order and runs the epilogue.
template <int KIND>
__global__ void __launch_bounds__(kMidWaves * 64)
gemm_mid_finish_kernel(GemmParams a, int NUG, int KS, const float* part) {
  __shared__ float rinv[16];
  const int b = (int)blockIdx.x;
  const int ug = b / kMidRT, mt = b - ug * kMidRT;
  if (ug >= NUG || mt * 16 >= a.M) return;  // uniform, before any barrier
  GemmMidFinish<KIND> f(a, rinv, ug, mt, KS, part);
  f.run();
}

template <int RT, int P, int KIND, int KS, bool NT = true>
__global__ void __launch_bounds__(kGemmWaves * 64)
    gemm_wide_kernel(GemmParams a, int NRG, int NUG, uint32_t* cnt, float* part) {
  extern __shared__ uint4 lds_dyn[];
  const int b = (int)blockIdx.x, q = b >> 3;
  const int j = q / (NRG * KS), rem = q - j * (NRG * KS);
  const int ks = rem / NRG, rg = rem - ks * NRG;
  const int ug = (b & 7) + 8 * j;
  if (ug >= NUG) return;  // uniform, before any barrier
  const int item = ug * NRG + rg;
  GemmWide<RT, P, KIND, KS, NT> g(a, *(GemmWideSmem<RT>*)lds_dyn, ug, rg, ks, KS > 1 ? cnt + item : nullptr,
                              KS > 1 ? part + (size_t)item * kWideItemFloats<RT, P> : nullptr);
  g.run();
}

// ---------------------------------------------------------------------------
// Verify attention.  Workgroup (chunk c, head h, request b): the R query rows
// of the request against keys [c*CK, min((c+1)*CK, L_b + R)); key j is
// visible to row i iff j <= L_b + i (causal inside the appended block).
// Scores: sixteen lanes share a key (HD/16 features each), four keys per wave
// step, and a reduce-scatter over the sixteen lanes leaves each row's dot
// product in one lane.  P V: each lane owns HD/64 output features.  Each
// chunk writes (max, sum, unnormalised output) per row for the combine
// kernel.
// ---------------------------------------------------------------------------
struct AttnParams {
  const float* q;
  const void* kc;
  const void* vc;
  const int32_t* lens;
  int b0, R, H, d, kv_stride;
  int Hkv, G;  // K/V heads of the cache; query head h reads K/V head h / G
  int CK, NC;
  int nb;  // requests of the call (bf16 kernels: the grid is one-dimensional)
  float scale;
  float* part_o;
  float* part_ml;
  uint32_t* cnt;
  int Rmax;
  void* act_out;
  size_t act_split;
};

// Raw K/V bytes of one lane: N features of a cache row, loaded as wide as
// their alignment allows, widened to float after the load has landed.
template <int N, bool KVBF16>
struct KVRaw {
  static constexpr int BYTES = N * (KVBF16 ? 2 : 4);
  static constexpr int WORDS = BYTES >= 4 ? BYTES / 4 : 1;
  uint32_t w[WORDS];
};

template <int N, bool KVBF16>
__device__ __forceinline__ void kv_load(KVRaw<N, KVBF16>& r, const void* base, size_t off) {
  constexpr int BYTES = KVRaw<N, KVBF16>::BYTES;
  const uint8_t* p = (const uint8_t*)base + off * (KVBF16 ? 2 : 4);
  if constexpr (BYTES >= 16) {
#pragma unroll
    for (int i = 0; i < BYTES / 16; ++i) {
      const uint4 v = *(const uint4*)(p + 16 * i);
      r.w[4 * i] = v.x;
      r.w[4 * i + 1] = v.y;
      r.w[4 * i + 2] = v.z;
      r.w[4 * i + 3] = v.w;
    }
  } else if constexpr (BYTES == 8) {
    const uint2 v = *(const uint2*)p;
    r.w[0] = v.x;
    r.w[1] = v.y;
  } else if constexpr (BYTES == 4) {
    r.w[0] = *(const uint32_t*)p;
  } else {
    r.w[0] = *(const uint16_t*)p;
  }
}

template <int N, bool KVBF16>
__device__ __forceinline__ void kv_zero(KVRaw<N, KVBF16>& r) {
#pragma unroll
  for (int i = 0; i < KVRaw<N, KVBF16>::WORDS; ++i) r.w[i] = 0u;
}

template <int N, bool KVBF16>
__device__ __forceinline__ float kv_get(const KVRaw<N, KVBF16>& r, int e) {
  if constexpr (KVBF16) {
    const uint32_t w = r.w[e >> 1];
    return (e & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
  } else {
    return __uint_as_float(r.w[e]);
  }
}

constexpr int kAttnKeysPerWave = kAttnChunk / 4;

template <int HD, int RMAX, bool KVBF16, bool ABF16>
__global__ void __launch_bounds__(256) attn_kernel(AttnParams p) {
  constexpr int DPL = HD / 16;  // VALU score phase (f32 cache): features per lane
  constexpr int DPV = HD / 64;  // VALU P V phase (f32 cache): features per lane
  constexpr int KPW = kAttnKeysPerWave;
  constexpr int FT = HD / 16;   // MFMA P V: feature tiles
  const int c = blockIdx.x, h = blockIdx.y, bl = blockIdx.z;
  const int bg = p.b0 + bl;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int R = p.R;
  const int L = p.lens[bg];
  const int nkeys = L + R;
  const int k_lo = c * kAttnChunk;
  const int k_hi = min(k_lo + kAttnChunk, nkeys);
  const int kw = k_lo + wave * KPW;  // this wave's first key
  const int g = lane >> 4, kl = lane & 15;

  __shared__ float s_lds[RMAX][kAttnChunk];
  __shared__ float o_lds[4][RMAX][HD];
  __shared__ float m_lds[RMAX], l_lds[RMAX];

  const size_t bh = (size_t)bl * p.H + h;
  float* po = p.part_o + ((bh * p.NC + c) * p.Rmax) * HD;
  float* pml = p.part_ml + ((bh * p.NC + c) * p.Rmax) * 2;
  // K blocks (k_cache_index; a float32 K cache: rows [key][HD])
  const size_t kbase = ((size_t)bg * p.Hkv + h / p.G) * p.kv_stride * HD;
  const size_t vbase = kbase;  // V blocks of kVBlock positions (v_cache_index, v_cache_index_f32)

  if (k_lo < k_hi) {
    if constexpr (KVBF16) {
      // -------- MFMA 16x16x32 bf16 for S = Q K^T and O = P V --------
      constexpr int KS = HD / 32;
      const uint16_t* kc = (const uint16_t*)p.kc;
      const uint16_t* vc = (const uint16_t*)p.vc;
      // loads first: K (B of S: 16 keys x 32 features per fragment) and V^T
      // (B of O: 32 keys x 16 features per fragment)
      uint4 kf[KPW / 16][KS];
#pragma unroll
      for (int grp = 0; grp < KPW / 16; ++grp) {
        const int key = kw + 16 * grp + kl;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          kf[grp][ks] = key < k_hi ? *(const uint4*)(kc + kbase + k_cache_index(32 * ks + 8 * g, key, HD))
                                   : make_uint4(0, 0, 0, 0);
      }
      uint4 vf[FT];
      const int kv0 = kw + 8 * g;  // first of this lane's 8 keys
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) {
        const uint16_t* vp = vc + vbase + v_cache_index(16 * ft + kl, kv0, HD);
        if (kv0 + 8 <= k_hi) {
          vf[ft] = *(const uint4*)vp;
        } else {
          uint32_t w[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t lo = (kv0 + 2 * e < k_hi) ? vp[2 * e] : 0u;
            const uint32_t hi = (kv0 + 2 * e + 1 < k_hi) ? vp[2 * e + 1] : 0u;
            w[e] = lo | (hi << 16);
          }
          vf[ft] = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
      uint4 qh[KS], ql[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        qh[ks] = make_uint4(0, 0, 0, 0);
        ql[ks] = make_uint4(0, 0, 0, 0);
      }
      if (kl < R) {
        const float* qp = p.q + (size_t)(bl * R + kl) * p.d + h * HD + 8 * g;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const float4 x0 = *(const float4*)(qp + 32 * ks);
          const float4 x1 = *(const float4*)(qp + 32 * ks + 4);
          const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
          uint32_t hw[4], lw[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint16_t h0 = f2bf(xs[2 * e]), h1 = f2bf(xs[2 * e + 1]);
            const uint16_t l0 = f2bf(xs[2 * e] - bf2f(h0)), l1 = f2bf(xs[2 * e + 1] - bf2f(h1));
            hw[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            lw[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
          }
          qh[ks] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
          ql[ks] = make_uint4(lw[0], lw[1], lw[2], lw[3]);
        }
      }
#pragma unroll
      for (int grp = 0; grp < KPW / 16; ++grp) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ql[ks]),
                                                        __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qh[ks]),
                                                        __builtin_bit_cast(bf16x8, kf[grp][ks]), acc, 0, 0, 0);
        }
        // D[i][j] sits in lane j + 16*(i/4), register i%4: rows 4g..4g+3 of key kl
        const int key = kw + 16 * grp + kl;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 4 * g + i;
          if (r < RMAX && key < k_hi) s_lds[r][key - k_lo] = (key <= L + r) ? acc[i] * p.scale : -INFINITY;
        }
      }
      __syncthreads();
      // chunk softmax, one wave per row; keys past the chunk end get p = 0
      const int nk = k_hi - k_lo;
      for (int r = wave; r < R; r += 4) {
        float mx = -INFINITY;
        for (int j = lane; j < nk; j += 64) mx = fmaxf(mx, s_lds[r][j]);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float sum = 0.f;
        for (int j = lane; j < kAttnChunk; j += 64) {
          const float e = (j < nk && mx != -INFINITY) ? expf(s_lds[r][j] - mx) : 0.f;
          s_lds[r][j] = e;
          sum += e;
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
        if (lane == 0) {
          m_lds[r] = mx;
          l_lds[r] = sum;
        }
      }
      __syncthreads();
      // O = P V: A = P rows (fp32 from LDS split into two bf16 terms) over the
      // wave's 32 keys, B = V^T fragments
      uint4 ph = make_uint4(0, 0, 0, 0), pl = make_uint4(0, 0, 0, 0);
      if (kl < R) {
        const float* pp = &s_lds[kl][kw - k_lo + 8 * g];
        const float4 x0 = *(const float4*)pp;
        const float4 x1 = *(const float4*)(pp + 4);
        const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        uint32_t hw[4], lw[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint16_t h0 = f2bf(xs[2 * e]), h1 = f2bf(xs[2 * e + 1]);
          const uint16_t l0 = f2bf(xs[2 * e] - bf2f(h0)), l1 = f2bf(xs[2 * e + 1] - bf2f(h1));
          hw[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
          lw[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        ph = make_uint4(hw[0], hw[1], hw[2], hw[3]);
        pl = make_uint4(lw[0], lw[1], lw[2], lw[3]);
      }
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pl), __builtin_bit_cast(bf16x8, vf[ft]),
                                                      acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ph), __builtin_bit_cast(bf16x8, vf[ft]),
                                                      acc, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 4 * g + i;
          if (r < RMAX) o_lds[wave][r][16 * ft + kl] = acc[i];
        }
      }
    } else {
      // -------- f32 cache: VALU --------
      constexpr int KSTEPS = KPW / 4;
      constexpr int RSH = (RMAX == 16) ? 0 : (RMAX == 8 ? 1 : 2);
      const float* kc = (const float*)p.kc;
      const float* vc = (const float*)p.vc;
      const int kg = lane >> 4, dg = lane & 15;
      float kr[KSTEPS][DPL];
#pragma unroll
      for (int s2 = 0; s2 < KSTEPS; ++s2) {
        const int k = kw + 4 * s2 + kg;
#pragma unroll
        for (int e = 0; e < DPL; e += 4) {
          float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
          if (k < k_hi) v = *(const float4*)(kc + kbase + (size_t)k * HD + dg * DPL + e);
          kr[s2][e] = v.x;
          kr[s2][e + 1] = v.y;
          kr[s2][e + 2] = v.z;
          kr[s2][e + 3] = v.w;
        }
      }
      float vt[DPV][KPW];  // V^T: this lane's features over the wave's keys
#pragma unroll
      for (int e = 0; e < DPV; ++e) {
        const float* vp = vc + vbase + v_cache_index_f32(lane * DPV + e, kw, HD);
#pragma unroll
        for (int j = 0; j < KPW; j += 4) {
          if (kw + j + 4 <= k_hi) {
            const float4 v = *(const float4*)(vp + j);
            vt[e][j] = v.x;
            vt[e][j + 1] = v.y;
            vt[e][j + 2] = v.z;
            vt[e][j + 3] = v.w;
          } else {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) vt[e][j + jj] = (kw + j + jj < k_hi) ? vp[j + jj] : 0.f;
          }
        }
      }
      float qr[RMAX][DPL];
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        if (r < R) {
          const float* qp = p.q + (size_t)(bl * R + r) * p.d + h * HD + dg * DPL;
#pragma unroll
          for (int e = 0; e < DPL; e += 4) {
            const float4 v = *(const float4*)(qp + e);
            qr[r][e] = v.x;
            qr[r][e + 1] = v.y;
            qr[r][e + 2] = v.z;
            qr[r][e + 3] = v.w;
          }
        } else {
#pragma unroll
          for (int e = 0; e < DPL; ++e) qr[r][e] = 0.f;
        }
      }
      const int rr = dg >> RSH;
      const bool writer = (dg & ((1 << RSH) - 1)) == 0 && rr < R;
#pragma unroll
      for (int s2 = 0; s2 < KSTEPS; ++s2) {
        const int k = kw + 4 * s2 + kg;
        float v[RMAX];
#pragma unroll
        for (int r = 0; r < RMAX; ++r) {
          float acc = 0.f;
#pragma unroll
          for (int e = 0; e < DPL; ++e) acc += qr[r][e] * kr[s2][e];
          v[r] = acc;
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const int off = 8 >> st;
          const int cur = RMAX >> st;
          if (cur > 1) {
            const int half = cur >> 1;
            const bool up = (dg & off) != 0;
#pragma unroll
            for (int j = 0; j < half; ++j) {
              const float mine = up ? v[half + j] : v[j];
              const float oth = up ? v[j] : v[half + j];
              v[j] = mine + __shfl_xor(oth, off);
            }
          } else {
            v[0] += __shfl_xor(v[0], off);
          }
        }
        if (k < k_hi && writer) s_lds[rr][k - k_lo] = (k <= L + rr) ? v[0] * p.scale : -INFINITY;
      }
      __syncthreads();
      const int nk = k_hi - k_lo;
      for (int r = wave; r < R; r += 4) {
        float mx = -INFINITY;
        for (int j = lane; j < nk; j += 64) mx = fmaxf(mx, s_lds[r][j]);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float sum = 0.f;
        for (int j = lane; j < kAttnChunk; j += 64) {
          const float e = (j < nk && mx != -INFINITY) ? expf(s_lds[r][j] - mx) : 0.f;
          s_lds[r][j] = e;
          sum += e;
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
        if (lane == 0) {
          m_lds[r] = mx;
          l_lds[r] = sum;
        }
      }
      __syncthreads();
      const int kk0 = kw - k_lo;
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        float a[DPV];
#pragma unroll
        for (int e = 0; e < DPV; ++e) a[e] = 0.f;
        if (r < R) {
#pragma unroll
          for (int j = 0; j < KPW; j += 4) {
            const float4 p4 = *(const float4*)&s_lds[r][kk0 + j];
#pragma unroll
            for (int e = 0; e < DPV; ++e)
              a[e] += p4.x * vt[e][j] + p4.y * vt[e][j + 1] + p4.z * vt[e][j + 2] + p4.w * vt[e][j + 3];
          }
#pragma unroll
          for (int e = 0; e < DPV; ++e) o_lds[wave][r][lane * DPV + e] = a[e];
        }
      }
    }
    __syncthreads();
    for (int idx = tid; idx < R * HD; idx += 256) {
      const int r = idx / HD, dd = idx % HD;
      po[r * HD + dd] = ((o_lds[0][r][dd] + o_lds[1][r][dd]) + o_lds[2][r][dd]) + o_lds[3][r][dd];
    }
    if (tid < R) {
      pml[tid * 2] = m_lds[tid];
      pml[tid * 2 + 1] = l_lds[tid];
    }
  } else if (tid < R) {
    pml[tid * 2] = -INFINITY;
    pml[tid * 2 + 1] = 0.f;
  }
}

// Merge of the chunk partials of every (request, head) in chunk order (a
// second launch: the kernel boundary orders the partial writes before these
// reads), written as the O-projection operand.
template <int HD, int RMAX, bool ABF16>
__global__ void __launch_bounds__(256) attn_combine_kernel(AttnParams p) {
  const int h = blockIdx.x, bl = blockIdx.y;
  const int tid = threadIdx.x;
  const int R = p.R;
  __shared__ float sc_lds[kAttnMaxChunks][RMAX];
  __shared__ float l_lds[kAttnMaxChunks][RMAX];
  const size_t bh = (size_t)bl * p.H + h;
  const float* po0 = p.part_o + (bh * p.NC * p.Rmax) * HD;
  const float* pml0 = p.part_ml + (bh * p.NC * p.Rmax) * 2;
  for (int idx = tid; idx < p.NC * R; idx += 256) {
    const int cc = idx / R, r = idx % R;
    const float2 ml = *(const float2*)(pml0 + ((size_t)cc * p.Rmax + r) * 2);
    sc_lds[cc][r] = ml.x;
    l_lds[cc][r] = ml.y;
  }
  __syncthreads();
  if (tid < R) {
    const int r = tid;
    float M = -INFINITY;
    for (int cc = 0; cc < p.NC; ++cc) M = fmaxf(M, sc_lds[cc][r]);
    float Ls = 0.f;
    for (int cc = 0; cc < p.NC; ++cc) {
      const float mc = sc_lds[cc][r];
      const float e = (mc == -INFINITY) ? 0.f : expf(mc - M);
      Ls += l_lds[cc][r] * e;
      sc_lds[cc][r] = e;
    }
    const float inv = 1.0f / Ls;
    for (int cc = 0; cc < p.NC; ++cc) sc_lds[cc][r] *= inv;
  }
  __syncthreads();
  for (int idx = tid; idx < R * HD; idx += 256) {
    const int r = idx / HD, dd = idx % HD;
    float O = 0.f;
#pragma unroll 8
    for (int cc = 0; cc < p.NC; ++cc) {
      const float sc = sc_lds[cc][r];
      const float v = po0[((size_t)cc * p.Rmax + r) * HD + dd];
      O += sc != 0.f ? v * sc : 0.f;
    }
    const int m = bl * R + r;
    store_act<ABF16>(p.act_out, p.act_split, (size_t)m * p.d + h * HD + dd, O);
  }
}

// Work of workgroup i of a bf16 attention launch over n_runs runs of chunks
// (one chunk each, or cpw) per (request, K/V head): run r, query head h,
// request bl.  The G query heads that share a K/V head get workgroups 8
// apart, which run on one XCD, so all but the first of their reads of the
// same keys and values can hit that XCD's L2.  ok == false: past the last
// item.
struct AttnWork {
  bool ok;
  int r, h, bl;
};
__device__ __forceinline__ AttnWork attn_work(int i, int n_runs, int Hkv, int G, int nb) {
  const int x = i & 7, j = i >> 3;     // XCD, slot on it
  const int t = j / G, g = j - t * G;  // group of 8 items, query head within the K/V head
  const int k = 8 * t + x;             // item: (run, K/V head, request), run fastest
  const int r = k % n_runs, q = k / n_runs;
  const int kvh = q % Hkv, bl = q / Hkv;
  return AttnWork{bl < nb, r, kvh * G + g, bl};
}
inline int attn_grid(int n_runs, int Hkv, int G, int nb) { return 8 * G * ((n_runs * Hkv * nb + 7) / 8); }

// bf16 cache, head_dim 128: chunks of CK keys, one 8-wave workgroup per
// (chunk, head, request) (device_attn.h; attn_work orders them); chunks past a
// request's last key exit at once, and the last chunk of a (request, head) to
// finish merges them into the O-projection operand.  The queries are staged in
// LDS and the V^T fragments loaded after the score products into the
// registers K held (attn_chunk_lr): 78 VGPRs, three workgroups per compute
// unit (keeping K, V and the queries in registers at once took 120: two).
template <bool ABF16, int CK, bool ARRIVE>
__global__ void __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(6)))
attn_lr_kernel(AttnParams p) {
  __shared__ AttnSmem<CK> sm;
  __shared__ AttnMergeSmem ms;
  __shared__ alignas(16) uint16_t sqh[kAttnRows][kAttnQPitch];
  __shared__ alignas(16) uint16_t sql[kAttnRows][kAttnQPitch];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const AttnWork wk = attn_work((int)blockIdx.x, p.NC, p.Hkv, p.G, p.nb);
  if (!wk.ok) return;
  const int bl = wk.bl, h = wk.h, bg = p.b0 + bl;
  const AttnItem it = attn_item<CK>(true, bl, h, wk.r, p.lens[bg], p.R, p.kc, p.vc,
                                    ((size_t)bg * p.Hkv + h / p.G) * p.kv_stride * kAttnHd);
  if (!it.active) return;  // past the request's last key: uniform, before any barrier
  // thread t stages features 4 (t % 32) .. + 3 of query row t / 32 (rows past R: zeros)
  const int qrow = tid >> 5, f4 = tid & 31;
  float4 qv = make_float4(0.f, 0.f, 0.f, 0.f);
  if (qrow < p.R) qv = *(const float4*)(p.q + (size_t)(bl * p.R + qrow) * p.d + h * kAttnHd + 4 * f4);
  uint4 kf[CK / 128][4];
  attn_load_k<CK>(it, wave, lane, kf);
  attn_stage_q(sqh, sql, qrow, 4 * f4, qv);
  __syncthreads();
  const floatx4 o = attn_chunk_lr<CK>(it, kf, sqh, sql, p.R, p.scale, sm);
  if constexpr (!ARRIVE) {  // attn_merge_kernel merges after this launch
    attn_publish<CK>(it, o, sm, p.part_o, p.part_ml, p.H, p.NC, p.Rmax, p.R);
    return;
  }
  attn_publish_merge<CK, false>(it, o, sm, ms, p.part_o, p.part_ml, p.cnt, p.H, p.NC, p.Rmax, p.R, [&](int oi, float O) {
    const int row = oi / kAttnHd, dd = oi - row * kAttnHd;
    store_act<ABF16>(p.act_out, p.act_split, (size_t)(bl * p.R + row) * p.d + h * kAttnHd + dd, O);
  });
}

// Grouped-query chunks: one workgroup per (chunk, K/V head, request) for all
// G query heads of the K/V head (attn_chunk_grp, T 16-row tiles of packed
// rows); the partials are merged by attn_merge_kernel.
template <bool ABF16, int T>
__global__ void __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(4)))
attn_g_kernel(AttnParams p) {
  constexpr int CK = kAttnChunkKeys;
  __shared__ AttnSmemG<CK, T> sm;
  __shared__ alignas(16) uint16_t sqh[16 * T][kAttnQPitch];
  __shared__ alignas(16) uint16_t sql[16 * T][kAttnQPitch];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const AttnWork wk = attn_work((int)blockIdx.x, p.NC, p.Hkv, 1, p.nb);
  if (!wk.ok) return;
  const int bl = wk.bl, kvh = wk.h, bg = p.b0 + bl;
  const AttnItem it = attn_item<CK>(true, bl, kvh, wk.r, p.lens[bg], p.R, p.kc, p.vc,
                                    ((size_t)bg * p.Hkv + kvh) * p.kv_stride * kAttnHd);
  if (!it.active) return;  // past the request's last key: uniform, before any barrier
  const int NR = p.G * p.R;
  // thread t stages features 4 (t % 32) .. + 3 of packed rows t / 32 + 16 j
  const int f4 = tid & 31;
  float4 qv[T];
  int gg[T][1], rw[T][1];
  attn_grp_rows<T, 1>(tid >> 5, p.R, gg, rw);
#pragma unroll
  for (int j = 0; j < T; ++j) {
    const int pr = (tid >> 5) + 16 * j;
    qv[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (pr < NR)
      qv[j] = *(const float4*)(p.q + (size_t)(bl * p.R + rw[j][0]) * p.d + (kvh * p.G + gg[j][0]) * kAttnHd + 4 * f4);
  }
  uint4 kf[CK / 128][4];
  attn_load_k<CK>(it, wave, lane, kf);
#pragma unroll
  for (int j = 0; j < T; ++j) attn_stage_q(sqh, sql, (tid >> 5) + 16 * j, 4 * f4, qv[j]);
  __syncthreads();
  floatx4 o[T];
  attn_chunk_grp<CK, T>(it, kf, sqh, sql, p.R, NR, p.scale, sm, o);
  attn_publish_grp<CK, T>(it, kvh, p.G, o, sm, p.part_o, p.part_ml, p.H, p.NC, p.Rmax, p.R);
}

// Second pass of the attention for launches with several rounds of chunk
// workgroups: workgroup (head h, request b) merges the chunk partials that
// attn_lr_kernel<..., false> stored (attn_merge, the same arithmetic as the
// last-arrival merge), so no chunk workgroup waits for its stores or an
// arrival counter while it holds its compute unit.
template <bool ABF16>
__global__ void __launch_bounds__(kAttnThreads) attn_merge_kernel(AttnParams p) {
  __shared__ AttnMergeSmem ms;
  const int h = blockIdx.x, bl = blockIdx.y, bg = p.b0 + bl;
  const int nc = (p.lens[bg] + p.R + kAttnChunkKeys - 1) / kAttnChunkKeys;
  attn_merge<false>((size_t)bl * p.H + h, nc, ms, p.part_o, p.part_ml, p.NC, p.Rmax, p.R, [&](int oi, float O) {
    const int row = oi / kAttnHd, dd = oi - row * kAttnHd;
    store_act<ABF16>(p.act_out, p.act_split, (size_t)(bl * p.R + row) * p.d + h * kAttnHd + dd, O);
  });
}

// Prefill attention of a forward with more than 16 rows per request
// (device_attn.h: attn_prefill_tiles): workgroup (group of W 16-row tiles,
// query head, request), one wave per tile.  Every tile group and query head
// of one (request, K/V head) runs on the same XCD, so that pair's keys and
// values, read by all of them, stay in one L2; on each XCD the groups with
// the most chunks start first.  Dynamic LDS: attn_prefill_dyn_bytes(W, NC).
template <bool ABF16, int W, int SK>
__global__ void __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(2)))
attn_prefill_kernel(AttnParams p, int ngrp) {
  __shared__ AttnPfSmem<W, SK> s;
  extern __shared__ uint4 lds_dyn[];
  const int i = blockIdx.x, x = i & 7, j = i >> 3;
  const int per = p.G * ngrp;
  const int pair = 8 * (j / per) + x, rem = j % per;
  if (pair >= p.nb * p.Hkv) return;
  const int gq = rem / ngrp, grp = ngrp - 1 - rem % ngrp;
  const int bl = pair / p.Hkv, kvh = pair % p.Hkv, h = kvh * p.G + gq, bg = p.b0 + bl;
  const size_t head_off = ((size_t)bg * p.Hkv + kvh) * p.kv_stride * kAttnHd;
  attn_prefill_tiles<W, SK>(s, (float2*)lds_dyn, p.NC, p.q + (size_t)bl * p.R * p.d, p.d, h,
                            (const uint16_t*)p.kc + head_off, (const uint16_t*)p.vc + head_off, p.lens[bg], p.R,
                            grp * W, p.scale, [&](int row, int dd, float O) {
                              store_act<ABF16>(p.act_out, p.act_split,
                                               (size_t)(bl * p.R + row) * p.d + h * kAttnHd + dd, O);
                            });
}

// ---------------------------------------------------------------------------
// Accept / reject and the correction draw (device_accept.h), one workgroup per
// request.
// ---------------------------------------------------------------------------
constexpr int kAcceptThreads = 1024;

__global__ void __launch_bounds__(kAcceptThreads) accept_kernel(AcceptParams p) {
  __shared__ AcceptSmem sm;
  accept_request<kAcceptThreads, false>(p, (int)blockIdx.x, sm);
}

// The correction draws of sampling requests over vocabulary slices: workgroup
// (slice, request), after accept_kernel (device_accept.h: correct_slice).
constexpr int kCorrThreads = 256;
constexpr int kCorrSliceTokens = 1024;  // tokens per slice (up to kCorrMaxSlices slices)

__global__ void __launch_bounds__(kCorrThreads) correct_kernel(AcceptParams p) {
  correct_slice<kCorrThreads>(p, (int)blockIdx.y, (int)blockIdx.x);
}

// ---------------------------------------------------------------------------
// Row softmax of logits / T (the draft side of Algorithm 1 keeps the
// distribution each of its tokens was drawn from): one workgroup per row,
// max then sum of exp in a fixed order, float32.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float block_reduce_256(float v, bool is_max, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float o = __shfl_xor(v, off);
    v = is_max ? fmaxf(v, o) : v + o;
  }
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < 4; ++w) r = is_max ? fmaxf(r, red[w]) : r + red[w];
  return r;
}

__global__ void __launch_bounds__(256) softmax_rows_kernel(const float* logits, int V, float invT, float* out) {
  __shared__ float red[4];
  const float* z = logits + (size_t)blockIdx.x * V;
  float* o = out + (size_t)blockIdx.x * V;
  float m = -INFINITY;
  for (int v = threadIdx.x; v < V; v += 256) m = fmaxf(m, z[v] * invT);
  m = block_reduce_256(m, true, red);
  float s = 0.f;
  for (int v = threadIdx.x; v < V; v += 256) s += expf(z[v] * invT - m);
  s = block_reduce_256(s, false, red);
  const float inv = 1.0f / s;
  for (int v = threadIdx.x; v < V; v += 256) o[v] = expf(z[v] * invT - m) * inv;
}

// ---------------------------------------------------------------------------
// Small kernels: commit, lens advance, packing.
// ---------------------------------------------------------------------------
// Context update m <- m + k + 1 with k clamped to the rows of the last verify
// call (k in [0, R - 1]); a k outside that range (a buffer the verify call did
// not write) is flagged.
__global__ void commit_kernel(int B, int R, int32_t* lens, int32_t* pending, const int32_t* n, const int32_t* corr,
                              uint32_t* err) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) {
    int k = n[b];
    if (k < 0 || k > R - 1) {
      flag_error(err, SPADE_DERR_COMMIT);
      k = k < 0 ? 0 : R - 1;
    }
    lens[b] += k + 1;
    pending[b] = corr[b];
  }
}

__global__ void copy_state_kernel(int B, int32_t* lens, int32_t* pending, const int32_t* src_lens,
                                  const int32_t* src_pending) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) {
    lens[b] = src_lens[b];
    pending[b] = src_pending[b];
  }
}

__global__ void advance_kernel(int b, int count, int32_t* lens, int32_t* pending, const int32_t* src) {
  if (threadIdx.x == 0) {
    lens[b] += count;
    if (src) pending[b] = *src;
  }
}

// Batched prefill.  A forward takes the next R prompt tokens of requests
// [b0, b0 + nb), each from the offset it has reached (its length now minus
// its length when the prefill began; 0 past its end: a placeholder row,
// written past its length); each length then advances by its real tokens;
// last, the pending tokens.
struct PrefillCounts {
  int n[64];
};

__global__ void prefill_counts_kernel(PrefillCounts c, int b0, int nb, int32_t* dst, const int32_t* lens,
                                      int32_t* base) {
  const int i = threadIdx.x;
  if (i < nb) {
    dst[b0 + i] = c.n[i];
    base[b0 + i] = lens[b0 + i];
  }
}

__global__ void prefill_gather_kernel(const int32_t* tokens, int ld, const int32_t* n_cache, const int32_t* base,
                                      const int32_t* lens, int b0, int nb, int R, int32_t* out) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= nb * R) return;
  const int b = b0 + m / R, pos = lens[b] - base[b] + m % R;
  out[m] = (pos >= 0 && pos < n_cache[b]) ? tokens[(size_t)b * ld + pos] : 0;
}

__global__ void prefill_advance_kernel(int b0, int nb, int R, const int32_t* n_cache, const int32_t* base,
                                       int32_t* lens) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nb) {
    const int b = b0 + i;
    const int rem = n_cache[b] - (lens[b] - base[b]);
    lens[b] += rem <= 0 ? 0 : (rem < R ? rem : R);
  }
}

__global__ void prefill_pending_kernel(int B, const int32_t* tokens, int ld, const int32_t* n_cache, int32_t* pending) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) pending[b] = tokens[(size_t)b * ld + n_cache[b]];
}

struct PackParams {
  const uint8_t* src;
  uint8_t* dst;
  int kind, wbf16;
  int N_src, row_off, K, NKB, n_units, pad_from, N_logical;
  int d, hd, F, dkv;
};

__global__ void pack_kernel(PackParams p) {
  const size_t chunk = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)p.n_units * p.NKB * 512;  // 16-byte chunks
  if (chunk >= total) return;
  const int lane = (int)(chunk & 63);
  const int j = (int)((chunk >> 6) & 7);
  const size_t t = chunk >> 9;
  const int kb = (int)(t % p.NKB);
  const int u = (int)(t / p.NKB);
  const int row = panel_row(p.kind, u, lane & 15, p.d, p.hd, p.F, p.dkv);
  const int g = lane >> 4;
  const int k = p.wbf16 ? kb * 256 + 32 * j + 8 * g : kb * 128 + 16 * j + 4 * g;
  const int srow = row - p.row_off;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (srow >= 0 && srow < p.N_src) {
    const size_t elt = p.wbf16 ? 2 : 4;
    v = *(const uint4*)(p.src + ((size_t)srow * p.K + k) * elt);
  } else if (!(p.row_off == 0 && row >= p.pad_from && row < p.N_logical)) {
    return;  // rows of another tensor sharing this matrix
  }
  *(uint4*)(p.dst + chunk * 16) = v;
}

// ---------------------------------------------------------------------------
// Host launchers.
// ---------------------------------------------------------------------------
namespace {

// The LDS operand copy needs more than the default dynamic LDS limit.
template <bool WBF16, int KIND>
hipError_t enable_lds_a() {
  static hipError_t once = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<WBF16, 1, true, KIND>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kGemmLdsABytes);
  return once;
}

template <bool WBF16, int KIND>
hipError_t launch_gemm_kind(const GemmParams& gp, int grid, int mt, hipStream_t st) {
  // activation operand copied to LDS once per workgroup where it fits
  const uint32_t lds = gemm_lds_a_bytes(gp.M, gp.act_stride, WBF16);
  if (mt == 1 && lds <= kGemmLdsABytes && gemm_lds_a_ok(gp.act_stride, WBF16)) {
    hipError_t e = enable_lds_a<WBF16, KIND>();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemm_kernel<WBF16, 1, true, KIND>), dim3(grid), dim3(kGemmWaves * 64), lds, st, gp);
  } else if (mt == 1) {
    hipLaunchKernelGGL((gemm_kernel<WBF16, 1, false, KIND>), dim3(grid), dim3(kGemmWaves * 64), 0, st, gp);
  } else {
    hipLaunchKernelGGL((gemm_kernel<WBF16, 2, false, KIND>), dim3(grid), dim3(kGemmWaves * 64), 0, st, gp);
  }
  return hipGetLastError();
}

template <bool WBF16>
hipError_t launch_gemm(int kind, const GemmParams& gp, int grid, int mt, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_gemm_kind<WBF16, GEMM_QKV>(gp, grid, mt, st);
    case GEMM_O: return launch_gemm_kind<WBF16, GEMM_O>(gp, grid, mt, st);
    case GEMM_GU: return launch_gemm_kind<WBF16, GEMM_GU>(gp, grid, mt, st);
    case GEMM_DOWN: return launch_gemm_kind<WBF16, GEMM_DOWN>(gp, grid, mt, st);
    default: return launch_gemm_kind<WBF16, GEMM_LM>(gp, grid, mt, st);
  }
}

template <int KS, int KIND>
hipError_t launch_split_ks(const GemmParams& gp, uint32_t* cnt, float* part, int G, hipStream_t st) {
  const void* fn = reinterpret_cast<const void*>(&gemm_split_kernel<KS, KIND>);
  static hipError_t attr =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)(kSplitSmemBytes + kGemmLdsABytes));
  if (attr != hipSuccess) return attr;
  const uint32_t lds = kSplitSmemBytes + gemm_split_lds_bytes(gp.M, gp.NKB, KS);
  hipLaunchKernelGGL((gemm_split_kernel<KS, KIND>), dim3(G * KS), dim3(kGemmWaves * 64), lds, st, gp, cnt, part, G);
  return hipGetLastError();
}

// k-splits for a bf16 projection with <= 16 rows whose whole operand does
// not fit in LDS, or whose panels are no more than the compute units: the
// fewest (2 or 4) whose split fits, with at most kSplitMaxGroups panel
// groups per workgroup; 0 when none qualifies (or the whole operand fits and
// the panels outnumber the compute units).  fixed > 0 forces that count
// where it qualifies.
int split_k_choice(const GemmParams& gp, int n_cu, int fixed) {
  if (gp.M > 16) return 0;
  const uint32_t whole = gemm_lds_a_bytes(gp.M, gp.act_stride, 1);
  const bool whole_fits = whole <= kGemmLdsABytes && gemm_lds_a_ok(gp.act_stride, 1);
  // an operand that fits one LDS copy needs no split, unless the panels are
  // too few for one per compute unit (the 7B O projection: 256 panels, one
  // 128 KB stream per workgroup; two k-splits: 3.520 -> 3.506 ms per 7B
  // batch-1 verify step)
  if (whole_fits && fixed <= 0 && gp.n_units > n_cu) return 0;
  for (int ks = 2; ks <= 4; ks *= 2) {
    if (fixed > 0 && ks != fixed) continue;
    const int G = n_cu / ks;
    if (G < 1) continue;
    const int groups = (gp.n_units + ks - 1) / ks;
    if ((groups + G - 1) / G > kSplitMaxGroups) continue;
    if (gemm_split_lds_bytes(gp.M, gp.NKB, ks) <= kGemmLdsABytes) return ks;
  }
  return 0;
}

}  // namespace

// Whether the LM head of a call with M rows leaves one statistics entry per
// row and panel (wide-row or split-K engine; the accept step then folds the
// panels in the skinny engine's workgroup order): the number of panels, else
// 0 (one entry per workgroup).  The same conditions as launch_layer_gemm.
int lm_stats_panels(spade_model md, int M) {
  const Dims& D = md->dims;
  if (D.wdt != SPADE_BF16) return 0;
  if (M > kWideMinRows) return md->wide_rt >= 0 ? D.Vpad / 16 : 0;
  if (md->split_ks < 0) return 0;
  GemmParams gp{};
  gp.M = M;
  gp.act_stride = D.d;
  gp.NKB = D.d / kblock_of(D.wdt);
  gp.n_units = D.Vpad / 16;
  return split_k_choice(gp, md->n_cu, md->split_ks) > 0 ? D.Vpad / 16 : 0;
}

namespace {

hipError_t launch_split(int kind, const GemmParams& gp, int ks, int n_cu, uint32_t* cnt, float* part, hipStream_t st) {
  const int G = n_cu / ks;
  if (ks == 2) {
    switch (kind) {
      case GEMM_QKV: return launch_split_ks<2, GEMM_QKV>(gp, cnt, part, G, st);
      case GEMM_O: return launch_split_ks<2, GEMM_O>(gp, cnt, part, G, st);
      case GEMM_GU: return launch_split_ks<2, GEMM_GU>(gp, cnt, part, G, st);
      case GEMM_DOWN: return launch_split_ks<2, GEMM_DOWN>(gp, cnt, part, G, st);
      default: return launch_split_ks<2, GEMM_LM>(gp, cnt, part, G, st);
    }
  }
  switch (kind) {
    case GEMM_QKV: return launch_split_ks<4, GEMM_QKV>(gp, cnt, part, G, st);
    case GEMM_O: return launch_split_ks<4, GEMM_O>(gp, cnt, part, G, st);
    case GEMM_GU: return launch_split_ks<4, GEMM_GU>(gp, cnt, part, G, st);
    case GEMM_DOWN: return launch_split_ks<4, GEMM_DOWN>(gp, cnt, part, G, st);
    default: return launch_split_ks<4, GEMM_LM>(gp, cnt, part, G, st);
  }
}

template <int RT, int P, int KIND, int KS, bool NT>
hipError_t launch_wide_nt(const GemmParams& gp, int nrg, int nug, uint32_t* cnt, float* part, hipStream_t st) {
  const void* fn = reinterpret_cast<const void*>(&gemm_wide_kernel<RT, P, KIND, KS, NT>);
  const uint32_t lds = gemm_wide_lds_bytes(RT);
  static hipError_t attr = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return attr;
  const int grid = 8 * ((nug + 7) / 8) * nrg * KS;
  hipLaunchKernelGGL((gemm_wide_kernel<RT, P, KIND, KS, NT>), dim3(grid), dim3(kGemmWaves * 64), lds, st, gp, nrg,
                     nug, cnt, part);
  return hipGetLastError();
}

// Non-temporal weight loads for launches of at most kWideNtRowGroups row
// groups (batched verification: 1-5); a many-row launch (prefill forwards:
// 32 and more row groups re-read every tile) keeps them in L2 (7B prefill
// down projection 256 -> 283 us per launch with them).  K-split launches
// are few-row ones.
constexpr int kWideNtRowGroups = 8;

template <int RT, int P, int KIND, int KS>
hipError_t launch_wide_rt(const GemmParams& gp, int nrg, int nug, uint32_t* cnt, float* part, hipStream_t st) {
  if constexpr (KS == 1)
    if (nrg > kWideNtRowGroups) return launch_wide_nt<RT, P, KIND, KS, false>(gp, nrg, nug, cnt, part, st);
  return launch_wide_nt<RT, P, KIND, KS, true>(gp, nrg, nug, cnt, part, st);
}

template <int KIND, int KS>
hipError_t launch_wide_ks(const GemmParams& gp, int rt, int p, int nrg, int nug, uint32_t* cnt, float* part,
                          hipStream_t st) {
  if constexpr (KS == 1) {
    if (p == 2 && rt == 3) return launch_wide_rt<3, 2, KIND, KS>(gp, nrg, nug, cnt, part, st);
  }
  if constexpr (KS != 2) {
    if (p == 2 && rt == 2) return launch_wide_rt<2, 2, KIND, KS>(gp, nrg, nug, cnt, part, st);
    if (rt == 3) return launch_wide_rt<3, 1, KIND, KS>(gp, nrg, nug, cnt, part, st);
  } else if (rt * p > 2) {
    return hipErrorInvalidValue;  // wide_choice gives two k-splits at most two accumulators
  }
  if (p == 2) return launch_wide_rt<1, 2, KIND, KS>(gp, nrg, nug, cnt, part, st);
  if (rt == 2) return launch_wide_rt<2, 1, KIND, KS>(gp, nrg, nug, cnt, part, st);
  return launch_wide_rt<1, 1, KIND, KS>(gp, nrg, nug, cnt, part, st);
}

template <int KIND>
hipError_t launch_wide_kind(const GemmParams& gp, int rt, int p, int ks, int nrg, int nug, uint32_t* cnt, float* part,
                            hipStream_t st) {
  if constexpr (KIND == GEMM_O || KIND == GEMM_DOWN) {
    if (ks == 4) return launch_wide_ks<KIND, 4>(gp, rt, p, nrg, nug, cnt, part, st);
    if (ks == 2) return launch_wide_ks<KIND, 2>(gp, rt, p, nrg, nug, cnt, part, st);
  }
  return launch_wide_ks<KIND, 1>(gp, rt, p, nrg, nug, cnt, part, st);
}

}  // namespace

// Published floats of a k-split wide launch of M rows and n_units panels
// with (rt, p): one block of kWideItemFloats per (unit group, row group).
size_t wide_split_floats(int n_units, int M, int rt, int p) {
  const size_t items = (size_t)gemm_wide_unit_groups(n_units, p) * gemm_wide_row_groups(M, rt);
  return items * (size_t)8 * kGemmWaves * p * rt * 256;
}

size_t mid_split_floats() { return (size_t)kMidItemFloats; }

// Rows above which a projection runs on the medium-M GEMM by default (the
// wide-row GEMM's time grows with the rows, the medium-M GEMM's barely).
int mid_min_rows(int kind) {
  switch (kind) {
    case GEMM_GU: return 112;
    case GEMM_O: return 128;
    case GEMM_DOWN: return 136;
    default: return kMidRT * 16;  // QKV, LM head: never
  }
}

// K-splits of a medium-M launch: the fewest that minimise the rounds of
// workgroups (one per compute unit at a time) times the k-blocks of the
// longest split, with a split launch charged about one and a half k-blocks
// for the range partials it adds to what the second pass reads back.  A
// fixed count (1-8) is used as given.
int mid_k_splits(int n_units, int NKB, int n_cu, int fixed_ks) {
  const int G = gemm_mid_unit_groups(n_units);
  if (fixed_ks > 0) return std::min(fixed_ks, kMidMaxSplits);
  int best = 1;
  double best_cost = -1.0;
  for (int ks = 1; ks <= kMidMaxSplits && ks <= NKB; ++ks) {
    int longest = 0;
    for (int s = 0; s < ks; ++s)
      longest = std::max(longest, NKB * (8 * (s + 1) / ks) / 8 - NKB * (8 * s / ks) / 8);
    const long rounds = ((long)G * ks + n_cu - 1) / n_cu;
    const double cost = (double)rounds * longest + (ks > 1 ? 1.5 : 0.0);
    if (best_cost < 0 || cost < best_cost - 1e-9) {
      best_cost = cost;
      best = ks;
    }
  }
  return best;
}

WideChoice wide_choice(int kind, int M, int n_units, int NKB, int K, int n_cu, int fixed_rt, int fixed_p, int fixed_ks,
                       size_t cap_items, size_t cap_floats) {
  const int tiles = (M + 15) / 16;
  const bool splittable = kind == GEMM_O || kind == GEMM_DOWN;
  const bool can_split = splittable && fixed_ks != 1;
  WideChoice best{1, 1, 1};
  double best_cost = -1.0, best_cu = 0.0;
  for (int p = 2; p >= 1; --p) {
    if (fixed_p > 0 && p != fixed_p) continue;
    for (int rt = 3; rt >= 1; --rt) {
      if (p == 2 && rt == 3 && splittable) continue;  // k-splittable kinds: not instantiated
      if (fixed_rt > 0 && rt != fixed_rt) continue;
      if (fixed_rt <= 0 && rt > tiles) continue;
      for (int ks = 1; ks <= 4; ks *= 2) {
        if (ks > 1 && !can_split) continue;
        if (fixed_ks > 1 && ks != fixed_ks && (can_split || ks != 1)) continue;
        // two k-splits hold three more range partials per accumulator: at most
        // two accumulators per lane (register budget)
        if (ks == 2 && rt * p > 2) continue;
        const int nug = gemm_wide_unit_groups(n_units, p), nrg = gemm_wide_row_groups(M, rt);
        const size_t items = (size_t)nug * nrg;
        if (ks > 1 && (items > cap_items || wide_split_floats(n_units, M, rt, p) > cap_floats)) continue;
        const long wgs = (long)items * ks;
        const long rounds = (wgs + n_cu - 1) / n_cu;
        const int nkbs = (NKB + ks - 1) / ks;
        double cost, cu = 0.0;
        if (!splittable) {
          // KB each workgroup moves per k-block, times rounds of workgroups
          cost = (double)rounds * (64 * p + 16 * rt);
        } else {
          // Fitted to stand-alone launches of the 7B and 33B O and down
          // projections at 144 and 28 rows over every tiling: per round a
          // workgroup streams its weight tiles at about 86 KB/us (75 with two
          // panels per wave), its operand k-blocks and published values at
          // 37 KB/us and pays 1.8 us of latency; all workgroups together stay
          // under 6 TB/s of HBM; the k-split combine (publish, arrive, the
          // last workgroup's reads and epilogue) adds about 10 us.
          const double slot_kb = 8.0 * rt * p;  // one published slot
          const double part_kb = ks > 1 ? (8.0 / ks + (9.0 - 8.0 / ks) / ks) * slot_kb : 0.0;
          const double w_kb = (double)nkbs * 64 * p, a_kb = (double)nkbs * 16 * rt + part_kb;
          const double per_round = w_kb / (p == 1 ? 86.0 : 75.0) + a_kb / 37.0 + 1.8;
          const double uniq_kb = (double)n_units * NKB * 8 + (double)M * K * 4 / 1024.0 +
                                 (ks > 1 ? items * (9.0 - 8.0 / ks) * slot_kb * 2 : 0.0);
          cu = rounds * per_round;
          cost = std::max(cu, uniq_kb / 6000.0 + 1.8) + (ks > 1 ? 10.0 : 0.0);
        }
        // ties (HBM-bound tilings) go to the least compute-unit time
        if (best_cost < 0 || cost < best_cost - 1e-9 || (cost <= best_cost + 1e-9 && cu < best_cu - 1e-9)) {
          best_cost = cost;
          best_cu = cu;
          best = WideChoice{rt, p, ks};
        }
      }
    }
  }
  // a fixed k-split that does not fit the published-value buffers: none
  if (best_cost < 0 && fixed_ks > 1)
    return wide_choice(kind, M, n_units, NKB, K, n_cu, fixed_rt, fixed_p, 1, cap_items, cap_floats);
  return best;
}

namespace {

// All rows of a bf16 projection in one launch.  Row tiles per workgroup,
// panels per wave and k-splits are fixed by the caller (> 0) or chosen by
// wide_choice: a compute unit streams about the same number of bytes per
// second whether they come from HBM or L2, so the time is close to the rounds
// of workgroups (one per compute unit at a time) times the bytes each moves
// per k-block, 64 KB of weights per panel per wave and 16 KB of operand per
// row tile; the O and down projections, which can also be k-split, use a
// model fitted to measured launches.
hipError_t launch_wide(spade_model md, int kind, const GemmParams& gp, hipStream_t st) {
  const Workspace& W = md->ws;
  const WideChoice c = wide_choice(kind, gp.M, gp.n_units, gp.NKB, gp.NKB * 256, md->n_cu, md->wide_rt, md->wide_p,
                                   md->wide_ks, W.wide_items, W.wide_floats);
  const int nug = gemm_wide_unit_groups(gp.n_units, c.p);
  const int nrg = gemm_wide_row_groups(gp.M, c.rt);
  switch (kind) {
    case GEMM_QKV: return launch_wide_kind<GEMM_QKV>(gp, c.rt, c.p, 1, nrg, nug, nullptr, nullptr, st);
    case GEMM_O: return launch_wide_kind<GEMM_O>(gp, c.rt, c.p, c.ks, nrg, nug, W.wide_cnt, W.wide_part, st);
    case GEMM_GU: return launch_wide_kind<GEMM_GU>(gp, c.rt, c.p, 1, nrg, nug, nullptr, nullptr, st);
    case GEMM_DOWN: return launch_wide_kind<GEMM_DOWN>(gp, c.rt, c.p, c.ks, nrg, nug, W.wide_cnt, W.wide_part, st);
    default: return launch_wide_kind<GEMM_LM>(gp, c.rt, c.p, 1, nrg, nug, nullptr, nullptr, st);
  }
}

hipError_t launch_attn_prefill(const AttnParams& ap, bool abf16, hipStream_t st) {
  constexpr int W = kPrefillAttnTiles, SK = kPrefillAttnKeys;
  const int most = (int)attn_prefill_dyn_bytes(W, kAttnMaxChunks);
  static hipError_t attr_b = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_prefill_kernel<true, W, SK>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, most);
  static hipError_t attr_f = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_prefill_kernel<false, W, SK>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, most);
  if (attr_b != hipSuccess) return attr_b;
  if (attr_f != hipSuccess) return attr_f;
  if (ap.NC > kAttnMaxChunks) return hipErrorInvalidValue;
  const int ngrp = ((ap.R + 15) / 16 + W - 1) / W;
  const dim3 grid(8 * ((ap.nb * ap.Hkv + 7) / 8) * ap.G * ngrp);
  const unsigned dyn = attn_prefill_dyn_bytes(W, ap.NC);
  if (abf16) hipLaunchKernelGGL((attn_prefill_kernel<true, W, SK>), grid, dim3(64 * W), dyn, st, ap, ngrp);
  else hipLaunchKernelGGL((attn_prefill_kernel<false, W, SK>), grid, dim3(64 * W), dyn, st, ap, ngrp);
  return hipGetLastError();
}

template <int KIND>
hipError_t launch_big_kind(const GemmParams& gp, hipStream_t st) {
  const void* fn = reinterpret_cast<const void*>(&gemm_big_kernel<KIND>);
  static hipError_t attr =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(GemmBigSmem));
  if (attr != hipSuccess) return attr;
  const int nrg = gemm_big_row_groups(gp.M), nug = gemm_big_unit_groups(gp.n_units);
  const int grid = 8 * ((nug + 7) / 8) * nrg;
  hipLaunchKernelGGL((gemm_big_kernel<KIND>), dim3(grid), dim3(kBigWaves * 64), sizeof(GemmBigSmem), st, gp, nrg,
                     nug);
  return hipGetLastError();
}

template <int KIND>
hipError_t launch_mid_kind(const GemmParams& gp, int ks, float* part, hipStream_t st) {
  const void* fn = reinterpret_cast<const void*>(&gemm_mid_kernel<KIND>);
  static hipError_t attr =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(GemmMidSmem));
  if (attr != hipSuccess) return attr;
  if (gp.M > kMidRT * 16 || ks < 1 || ks > kMidMaxSplits) return hipErrorInvalidValue;
  const int nug = gemm_mid_unit_groups(gp.n_units);
  hipLaunchKernelGGL((gemm_mid_kernel<KIND>), dim3(nug * ks), dim3(kMidWaves * 64), sizeof(GemmMidSmem), st, gp, nug,
                     ks, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gemm_mid_finish_kernel<KIND>), dim3(nug * kMidRT), dim3(kMidWaves * 64), 0, st, gp, nug, ks,
                     (const float*)part);
  return hipGetLastError();
}

hipError_t launch_mid(int kind, const GemmParams& gp, int ks, float* part, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_mid_kind<GEMM_QKV>(gp, ks, part, st);
    case GEMM_O: return launch_mid_kind<GEMM_O>(gp, ks, part, st);
    case GEMM_GU: return launch_mid_kind<GEMM_GU>(gp, ks, part, st);
    case GEMM_DOWN: return launch_mid_kind<GEMM_DOWN>(gp, ks, part, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_big(int kind, const GemmParams& gp, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_big_kind<GEMM_QKV>(gp, st);
    case GEMM_O: return launch_big_kind<GEMM_O>(gp, st);
    case GEMM_GU: return launch_big_kind<GEMM_GU>(gp, st);
    case GEMM_DOWN: return launch_big_kind<GEMM_DOWN>(gp, st);
    default: return hipErrorInvalidValue;
  }
}

template <int HD, int RMAX>
hipError_t launch_attn_r(const AttnParams& ap, bool kvbf16, bool abf16, dim3 grid, hipStream_t st) {
  if (kvbf16 && abf16) hipLaunchKernelGGL((attn_kernel<HD, RMAX, true, true>), grid, dim3(256), 0, st, ap);
  else if (kvbf16) hipLaunchKernelGGL((attn_kernel<HD, RMAX, true, false>), grid, dim3(256), 0, st, ap);
  else if (abf16) hipLaunchKernelGGL((attn_kernel<HD, RMAX, false, true>), grid, dim3(256), 0, st, ap);
  else hipLaunchKernelGGL((attn_kernel<HD, RMAX, false, false>), grid, dim3(256), 0, st, ap);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 cgrid(grid.y, grid.z);
  if (abf16) hipLaunchKernelGGL((attn_combine_kernel<HD, RMAX, true>), cgrid, dim3(256), 0, st, ap);
  else hipLaunchKernelGGL((attn_combine_kernel<HD, RMAX, false>), cgrid, dim3(256), 0, st, ap);
  return hipGetLastError();
}

template <int HD>
hipError_t launch_attn_hd(const AttnParams& ap, bool kvbf16, bool abf16, dim3 grid, hipStream_t st) {
  if (ap.R <= 4) return launch_attn_r<HD, 4>(ap, kvbf16, abf16, grid, st);
  if (ap.R <= 8) return launch_attn_r<HD, 8>(ap, kvbf16, abf16, grid, st);
  return launch_attn_r<HD, 16>(ap, kvbf16, abf16, grid, st);
}

}  // namespace

hipError_t launch_layer_gemm(spade_model md, spade_kv kv, int kind, int layer, const ForwardCall& fc,
                             hipStream_t st) {
  const Dims& D = md->dims;
  const Workspace& W = md->ws;
  const bool wb = D.wdt == SPADE_BF16;
  const int KBd = kblock_of(D.wdt);
  const size_t kv_layer = (size_t)kv->max_batch * D.KVH * kv->stride * D.hd;  // elements
  const size_t kv_elt = D.kvdt == SPADE_BF16 ? 2 : 4;
  const uint8_t* lb = md->weights + (size_t)layer * md->lay.layer_bytes;
  const int M = fc.nb * fc.R;

  GemmParams g{};
  g.R = fc.R;
  g.b0 = fc.b0;
  g.lens = kv->lens;
  g.inv_din = 1.0f / (float)D.d;
  g.eps = D.eps;
  g.n_ssq = D.d / 16;
  g.H = D.H;
  g.Hkv = D.KVH;
  g.hd = D.hd;
  g.d = D.d;
  g.F = D.F;
  g.kv_stride = kv->stride;
  g.kv_bf16 = D.kvdt == SPADE_BF16;
  g.kv_bytes = (uint32_t)(kv_layer * kv_elt);
  g.rope = W.rope;
  g.x = W.x;
  g.V = D.V;
  g.err = W.err;
  const uint8_t* wmat;
  int K, units;
  const void* act;
  size_t act_split;
  switch (kind) {
    case GEMM_QKV:
      wmat = lb + md->lay.qkv; K = D.d; units = (D.d + 2 * D.dkv) / 16; act = W.act_n; act_split = W.act_split;
      g.ssq_in = W.ssq;
      g.q_out = W.q;
      g.kc = kv->k + (size_t)layer * kv_layer * kv_elt;
      g.vc = kv->v + (size_t)layer * kv_layer * kv_elt;
      break;
    case GEMM_O:
      // O projection + residual; operand of gate/up = x * g_ffn
      wmat = lb + md->lay.o; K = D.d; units = D.d / 16; act = W.act_o; act_split = W.act_split;
      g.act_out = W.act_n;
      g.act_out_split = W.act_split;
      g.act_out_stride = D.d;
      g.g_next = (const float*)(lb + md->lay.g_ffn);
      g.ssq_out = W.ssq;
      g.n_ssq_out = D.d / 16;
      break;
    case GEMM_GU:
      wmat = lb + md->lay.gu; K = D.d; units = 2 * D.F / 16; act = W.act_n; act_split = W.act_split;
      g.ssq_in = W.ssq;
      g.act_out = W.act_f;
      g.act_out_split = W.actf_split;
      g.act_out_stride = D.F;
      break;
    case GEMM_DOWN:
      // down + residual; operand of the next layer (or of the LM head)
      wmat = lb + md->lay.down; K = D.F; units = D.d / 16; act = W.act_f; act_split = W.actf_split;
      g.act_out = W.act_n;
      g.act_out_split = W.act_split;
      g.act_out_stride = D.d;
      g.g_next = (layer + 1 < D.L)
                     ? (const float*)(md->weights + (size_t)(layer + 1) * md->lay.layer_bytes + md->lay.g_attn)
                     : (const float*)(md->weights + md->lay.g_final);
      g.ssq_out = W.ssq;
      g.n_ssq_out = D.d / 16;
      break;
    default:  // GEMM_LM
      wmat = md->weights + md->lay.lm; K = D.d; units = D.Vpad / 16; act = W.act_n; act_split = W.act_split;
      g.ssq_in = W.ssq;
      g.logits = fc.logits_out;
      g.stats = W.stats;
      g.pstats = W.stats;  // per-panel layout when the wide-row or split-K engine runs it
      g.mode = fc.mode;
      g.inv_T = fc.inv_T;
      g.have_q = fc.have_q;
      break;
  }
  const int grid = std::min(units, md->gemm_wgs);
  g.NU = grid;  // LM head: one statistics entry per workgroup and row
  if (wb && M > kWideMinRows && kind != GEMM_LM && md->big_gemm != 1) {
    // many rows (prefill): 128-row x 256-column workgroups, once there are
    // enough of them to fill the chip (or always, when forced)
    const long wgs = (long)gemm_big_row_groups(M) * gemm_big_unit_groups(units);
    if (md->big_gemm == 2 || wgs >= md->n_cu) {
      GemmParams gp = g;
      gp.w = wmat;
      gp.NKB = K / KBd;
      gp.n_units = units;
      gp.M = M;
      gp.m0 = 0;
      gp.act = act;
      gp.act_split = act_split;
      gp.act_stride = K;
      return launch_big(kind, gp, st);
    }
  }
  // batched verification: every row in one workgroup per panel group (by
  // default the gate/up projection of more than 112 rows, O and down of
  // more than 128 and 136: the crossovers with the wide-row GEMM measured at
  // the 7B shape; the QKV projection measured no faster)
  if (wb && M > kWideMinRows && M <= kMidRT * 16 && kind != GEMM_LM && md->mid_gemm != 1 &&
      (md->mid_gemm == 2 || M > mid_min_rows(kind)) && W.mid_part && (size_t)gemm_mid_unit_groups(units) <= W.mid_items) {
    GemmParams gp = g;
    gp.w = wmat;
    gp.NKB = K / KBd;
    gp.n_units = units;
    gp.M = M;
    gp.m0 = 0;
    gp.act = act;
    gp.act_split = act_split;
    gp.act_stride = K;
    const int ks = mid_k_splits(units, gp.NKB, md->n_cu, md->mid_ks);
    return launch_mid(kind, gp, ks, W.mid_part, st);
  }
  if (wb && M > kWideMinRows && md->wide_rt >= 0) {
    // batched rows: every row in one launch, weights streamed once
    GemmParams gp = g;
    gp.w = wmat;
    gp.NKB = K / KBd;
    gp.n_units = units;
    gp.M = M;
    gp.m0 = 0;
    gp.act = act;
    gp.act_split = act_split;
    gp.act_stride = K;
    return launch_wide(md, kind, gp, st);
  }
  for (int m0 = 0; m0 < M; m0 += kMaxRowsPerGemm) {
    GemmParams gp = g;
    gp.w = wmat;
    gp.NKB = K / KBd;
    gp.n_units = units;
    gp.M = std::min(kMaxRowsPerGemm, M - m0);
    gp.m0 = m0;
    gp.act = act;
    gp.act_split = act_split;
    gp.act_stride = K;
    const int mt = gp.M > 16 ? 2 : 1;
    // (the LM head only for a call of <= 16 rows in all: lm_stats_panels)
    if (wb && md->split_ks >= 0 && (kind != GEMM_LM || M <= kWideMinRows)) {
      const int ks = split_k_choice(gp, md->n_cu, md->split_ks);
      if (ks > 0) {
        hipError_t r = launch_split(kind, gp, ks, md->n_cu, W.split_cnt, W.split_part, st);
        if (r != hipSuccess) return r;
        continue;
      }
    }
    hipError_t r = wb ? launch_gemm<true>(kind, gp, grid, mt, st) : launch_gemm<false>(kind, gp, grid, mt, st);
    if (r != hipSuccess) return r;
  }
  return hipSuccess;
}

hipError_t launch_forward(spade_model md, spade_kv kv, const ForwardCall& fc, hipStream_t st) {
  const Dims& D = md->dims;
  const Workspace& W = md->ws;
  const bool wb = D.wdt == SPADE_BF16;
  const int M = fc.nb * fc.R;
  hipError_t e;

  EmbedParams ep{};
  ep.E = md->weights + md->lay.embed;
  ep.g = (const float*)(md->weights + md->lay.g_attn);  // layer 0
  ep.tokens = fc.tokens;
  ep.drafts = fc.drafts;
  ep.pending = kv->pending;
  ep.b0 = fc.b0;
  ep.R = fc.R;
  ep.d = D.d;
  ep.V = D.V;
  ep.x = W.x;
  ep.act = W.act_n;
  ep.act_split = W.act_split;
  ep.ssq = W.ssq;
  ep.err = W.err;
  ep.lens = kv->lens;

  const size_t kv_layer = (size_t)kv->max_batch * D.KVH * kv->stride * D.hd;  // elements
  const size_t kv_elt = D.kvdt == SPADE_BF16 ? 2 : 4;

  // attention chunks over the longest request: for a bf16 cache with
  // head_dim 128 the 8-wave MFMA kernel, else kAttnChunk
  int max_keys = 0;
  for (int b = fc.b0; b < fc.b0 + fc.nb; ++b) max_keys = std::max(max_keys, kv->lens_ub[b] + fc.R);
  const bool tiled = D.kvdt == SPADE_BF16 && D.hd == kAttnHd;
  const bool mfma_attn = tiled && fc.R <= kAttnRows;
  // more rows per request than one verify call: the prefill attention
  const bool prefill_attn = fc.R > kAttnRows;
  if (prefill_attn && (!tiled || fc.tokens == nullptr || fc.want_logits)) return hipErrorInvalidValue;
  const int CK = tiled ? kAttnChunkKeys : kAttnChunk;
  const int NC = (max_keys + CK - 1) / CK;
  if (NC > W.NCmax || NC > kAttnMaxChunks) return hipErrorInvalidValue;
  // every request's keys must fit the cache and the chunks launched below
  ep.len_limit = std::min(kv->max_len, NC * CK);
  // one workgroup per (row, 256 columns)
  const dim3 egrid(M, (D.d + 255) / 256);
  if (wb) hipLaunchKernelGGL(embed_kernel<true>, egrid, dim3(256), 0, st, ep);
  else hipLaunchKernelGGL(embed_kernel<false>, egrid, dim3(256), 0, st, ep);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // one chunk per workgroup: merge by the last chunk to arrive, or, when the
  // call has at least four chunks per compute unit (several rounds of chunk
  // workgroups), in a second launch (measured: C4 12.78 -> 12.25 ms, C5
  // 17.66 -> 17.49; at C2 the extra launch costs more than it saves)
  bool two_pass = false;
  if (md->attn_merge == 2) {
    two_pass = true;
  } else if (md->attn_merge == 0) {
    long chunks = 0;
    for (int b = fc.b0; b < fc.b0 + fc.nb; ++b) chunks += (kv->lens_ub[b] + fc.R + CK - 1) / CK;
    two_pass = chunks * D.H >= 4L * md->n_cu;
  }

  for (int l = 0; l < D.L; ++l) {
    if ((e = launch_layer_gemm(md, kv, GEMM_QKV, l, fc, st)) != hipSuccess) return e;
    AttnParams ap{};
    ap.q = W.q;
    ap.kc = kv->k + (size_t)l * kv_layer * kv_elt;
    ap.vc = kv->v + (size_t)l * kv_layer * kv_elt;
    ap.lens = kv->lens;
    ap.b0 = fc.b0;
    ap.R = fc.R;
    ap.H = D.H;
    ap.Hkv = D.KVH;
    ap.G = D.H / D.KVH;
    ap.d = D.d;
    ap.kv_stride = kv->stride;
    ap.CK = CK;
    ap.NC = NC;
    ap.scale = 1.0f / sqrtf((float)D.hd);
    ap.part_o = W.attn_o;
    ap.part_ml = W.attn_ml;
    ap.cnt = W.attn_cnt;
    ap.Rmax = W.Rmax;
    ap.act_out = W.act_o;
    ap.act_split = W.act_split;
    const dim3 agrid(NC, D.H, fc.nb);
    const bool kvb = D.kvdt == SPADE_BF16;
    ap.nb = fc.nb;
    if (prefill_attn) {
      e = launch_attn_prefill(ap, wb, st);
    } else if (mfma_attn && two_pass) {
      // grouped-query models: one workgroup per K/V head and chunk for the
      // G query heads when their G R rows fit three 16-row tiles (8B-GQA
      // batched: 13.42 -> 13.09 ms)
      const int G = D.H / D.KVH, T = (G * fc.R + 15) / 16;
      if (md->attn_grouped == 0 && G > 1 && T <= 3) {
        const dim3 ggrid(attn_grid(NC, D.KVH, 1, fc.nb));
        if (T == 1) {
          if (wb) hipLaunchKernelGGL((attn_g_kernel<true, 1>), ggrid, dim3(kAttnThreads), 0, st, ap);
          else hipLaunchKernelGGL((attn_g_kernel<false, 1>), ggrid, dim3(kAttnThreads), 0, st, ap);
        } else if (T == 2) {
          if (wb) hipLaunchKernelGGL((attn_g_kernel<true, 2>), ggrid, dim3(kAttnThreads), 0, st, ap);
          else hipLaunchKernelGGL((attn_g_kernel<false, 2>), ggrid, dim3(kAttnThreads), 0, st, ap);
        } else {
          if (wb) hipLaunchKernelGGL((attn_g_kernel<true, 3>), ggrid, dim3(kAttnThreads), 0, st, ap);
          else hipLaunchKernelGGL((attn_g_kernel<false, 3>), ggrid, dim3(kAttnThreads), 0, st, ap);
        }
      } else {
        const dim3 bgrid(attn_grid(NC, D.KVH, D.H / D.KVH, fc.nb));
        if (wb) hipLaunchKernelGGL((attn_lr_kernel<true, kAttnChunkKeys, false>), bgrid, dim3(kAttnThreads), 0, st, ap);
        else hipLaunchKernelGGL((attn_lr_kernel<false, kAttnChunkKeys, false>), bgrid, dim3(kAttnThreads), 0, st, ap);
      }
      if ((e = hipGetLastError()) != hipSuccess) return e;
      if (wb) hipLaunchKernelGGL((attn_merge_kernel<true>), dim3(D.H, fc.nb), dim3(kAttnThreads), 0, st, ap);
      else hipLaunchKernelGGL((attn_merge_kernel<false>), dim3(D.H, fc.nb), dim3(kAttnThreads), 0, st, ap);
      e = hipGetLastError();
    } else if (mfma_attn) {
      const dim3 bgrid(attn_grid(NC, D.KVH, D.H / D.KVH, fc.nb));
      if (wb) hipLaunchKernelGGL((attn_lr_kernel<true, kAttnChunkKeys, true>), bgrid, dim3(kAttnThreads), 0, st, ap);
      else hipLaunchKernelGGL((attn_lr_kernel<false, kAttnChunkKeys, true>), bgrid, dim3(kAttnThreads), 0, st, ap);
      e = hipGetLastError();
    } else if (D.hd == 64) {
      e = launch_attn_hd<64>(ap, kvb, wb, agrid, st);
    } else {
      e = launch_attn_hd<128>(ap, kvb, wb, agrid, st);
    }
    if (e != hipSuccess) return e;
    if ((e = launch_layer_gemm(md, kv, GEMM_O, l, fc, st)) != hipSuccess) return e;
    if ((e = launch_layer_gemm(md, kv, GEMM_GU, l, fc, st)) != hipSuccess) return e;
    if ((e = launch_layer_gemm(md, kv, GEMM_DOWN, l, fc, st)) != hipSuccess) return e;
  }
  if (fc.want_logits)
    if ((e = launch_layer_gemm(md, kv, GEMM_LM, 0, fc, st)) != hipSuccess) return e;
  return hipSuccess;
}

hipError_t launch_accept(spade_model md, const AcceptCall& ac, hipStream_t st) {
  AcceptParams p{};
  p.logits = ac.logits;
  p.stats = ac.stats;
  p.NU = ac.NU;
  p.panels = ac.panels;
  p.B = ac.B;
  p.V = ac.V;
  p.gamma = ac.gamma;
  p.R = ac.gamma + 1;
  p.drafts = ac.drafts;
  p.q = ac.q;
  p.u = ac.u;
  p.mode = ac.mode;
  p.inv_T = ac.inv_T;
  p.n_out = ac.n_out;
  p.corr_out = ac.corr_out;
  p.err = md->ws.err;
  // a request may sample: its correction draw (a pass over the vocabulary
  // with two logarithms per token) goes to a second launch over slices of
  // the vocabulary, unless turned off (the accept workgroup then draws it)
  const bool may_sample = ac.u != nullptr && (ac.q != nullptr || ac.gamma == 0);
  const bool split = may_sample && md->corr_split != 1 && ac.B <= md->max_batch;
  if (split) {
    p.corr_slices = std::min(kCorrMaxSlices, (ac.V + kCorrSliceTokens - 1) / kCorrSliceTokens);
    p.corr_lse = md->ws.corr_lse;
    p.corr_part = md->ws.corr_part;
    p.corr_cnt = md->ws.corr_cnt;
  }
  hipLaunchKernelGGL(accept_kernel, dim3(ac.B), dim3(kAcceptThreads), 0, st, p);
  if (split) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(correct_kernel, dim3(p.corr_slices, ac.B), dim3(kCorrThreads), 0, st, p);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scratch of spade_accept_from_logits_noalloc, for callers that cannot
// allocate: the sliced correction draw's per-request arrival counters,
// log-sum-exps and per-slice winners for up to kNoAllocMaxB requests, in a
// file-scope device array.  Each device holds its own copy at its own
// address (looked up once per device); every call on a device uses that copy,
// so calls that overlap on one device race.  The accept kernel zeroes a
// request's counter before the correction launch uses it.
// ---------------------------------------------------------------------------
struct NoAllocScratch {
  uint32_t cnt[kNoAllocMaxB];
  float lse[kNoAllocMaxB];
  float part[kNoAllocMaxB * kCorrMaxSlices * 4];
};
static __device__ __align__(256) uint8_t scratch[sizeof(NoAllocScratch)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (the host symbol is a
// stand-in, never a device address).
hipError_t scratch_address(uint8_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = (uint8_t*)g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

size_t noalloc_scratch_bytes() { return sizeof(NoAllocScratch); }

hipError_t launch_accept_noalloc(const AcceptCall& ac, uint32_t* err, hipStream_t st) {
  uint8_t* base = nullptr;
  hipError_t e = scratch_address(&base);
  if (e != hipSuccess) return e;
  AcceptParams p{};
  p.logits = ac.logits;
  p.stats = nullptr;
  p.B = ac.B;
  p.V = ac.V;
  p.gamma = ac.gamma;
  p.R = ac.gamma + 1;
  p.drafts = ac.drafts;
  p.q = ac.q;
  p.u = ac.u;
  p.mode = ac.mode;
  p.inv_T = ac.inv_T;
  p.n_out = ac.n_out;
  p.corr_out = ac.corr_out;
  p.err = err;
  // a call that may sample draws its corrections over vocabulary slices,
  // with this device's scratch
  const bool may_sample = ac.u != nullptr && (ac.q != nullptr || ac.gamma == 0);
  if (may_sample) {
    p.corr_slices = std::min(kCorrMaxSlices, (ac.V + kCorrSliceTokens - 1) / kCorrSliceTokens);
    p.corr_cnt = (uint32_t*)(base + offsetof(NoAllocScratch, cnt));
    p.corr_lse = (float*)(base + offsetof(NoAllocScratch, lse));
    p.corr_part = (float*)(base + offsetof(NoAllocScratch, part));
  }
  hipLaunchKernelGGL(accept_kernel, dim3(ac.B), dim3(kAcceptThreads), 0, st, p);
  if (may_sample) {
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(correct_kernel, dim3(p.corr_slices, ac.B), dim3(kCorrThreads), 0, st, p);
  }
  return hipGetLastError();
}

hipError_t launch_pack(spade_model md, int kind, int layer, const void* src, hipStream_t st) {
  const Dims& D = md->dims;
  const bool wb = D.wdt == SPADE_BF16;
  const size_t elt = wb ? 2 : 4;
  const uint8_t* lb = md->weights + (size_t)layer * md->lay.layer_bytes;
  uint8_t* dst = nullptr;
  PackParams pp{};
  pp.src = (const uint8_t*)src;
  pp.wbf16 = wb;
  pp.d = D.d;
  pp.hd = D.hd;
  pp.F = D.F;
  pp.dkv = D.dkv;
  switch (kind) {
    case SPADE_WQ: case SPADE_WK: case SPADE_WV:
      pp.kind = GEMM_QKV; pp.K = D.d;
      pp.N_src = kind == SPADE_WQ ? D.d : D.dkv;
      pp.row_off = kind == SPADE_WQ ? 0 : (kind == SPADE_WK ? D.d : D.d + D.dkv);
      pp.N_logical = D.d + 2 * D.dkv; pp.n_units = pp.N_logical / 16; dst = (uint8_t*)lb + md->lay.qkv; break;
    case SPADE_WO:
      pp.kind = GEMM_O; pp.K = D.d; pp.N_src = D.d; pp.row_off = 0; pp.N_logical = D.d;
      pp.n_units = D.d / 16; dst = (uint8_t*)lb + md->lay.o; break;
    case SPADE_WGATE: case SPADE_WUP:
      pp.kind = GEMM_GU; pp.K = D.d; pp.N_src = D.F; pp.row_off = (kind - SPADE_WGATE) * D.F;
      pp.N_logical = 2 * D.F; pp.n_units = 2 * D.F / 16; dst = (uint8_t*)lb + md->lay.gu; break;
    case SPADE_WDOWN:
      pp.kind = GEMM_DOWN; pp.K = D.F; pp.N_src = D.d; pp.row_off = 0; pp.N_logical = D.d;
      pp.n_units = D.d / 16; dst = (uint8_t*)lb + md->lay.down; break;
    case SPADE_LM_HEAD:
      pp.kind = GEMM_LM; pp.K = D.d; pp.N_src = D.V; pp.row_off = 0; pp.N_logical = D.Vpad;
      pp.n_units = D.Vpad / 16; dst = md->weights + md->lay.lm; break;
    case SPADE_EMBED:
      return hipMemcpyAsync(md->weights + md->lay.embed, src, (size_t)D.V * D.d * elt, hipMemcpyDeviceToDevice, st);
    case SPADE_G_ATTN:
      return hipMemcpyAsync((uint8_t*)lb + md->lay.g_attn, src, (size_t)D.d * 4, hipMemcpyDeviceToDevice, st);
    case SPADE_G_FFN:
      return hipMemcpyAsync((uint8_t*)lb + md->lay.g_ffn, src, (size_t)D.d * 4, hipMemcpyDeviceToDevice, st);
    case SPADE_G_FINAL:
      return hipMemcpyAsync(md->weights + md->lay.g_final, src, (size_t)D.d * 4, hipMemcpyDeviceToDevice, st);
    default:
      return hipErrorInvalidValue;
  }
  pp.dst = dst;
  pp.pad_from = kind == SPADE_LM_HEAD ? D.V : pp.N_logical;
  pp.NKB = pp.K / kblock_of(D.wdt);
  const size_t total = (size_t)pp.n_units * pp.NKB * 512;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL(pack_kernel, dim3(blocks), dim3(256), 0, st, pp);
  return hipGetLastError();
}

hipError_t launch_softmax(const float* logits, int rows, int V, float invT, float* out, hipStream_t st) {
  hipLaunchKernelGGL(softmax_rows_kernel, dim3(rows), dim3(256), 0, st, logits, V, invT, out);
  return hipGetLastError();
}

hipError_t launch_commit(spade_kv kv, int B, int R, const int32_t* n, const int32_t* corr, hipStream_t st) {
  hipLaunchKernelGGL(commit_kernel, dim3((B + 63) / 64), dim3(64), 0, st, B, R, kv->lens, kv->pending, n, corr,
                     kv->model->ws.err);
  return hipGetLastError();
}

hipError_t launch_copy_state(int B, int32_t* lens, int32_t* pending, const int32_t* src_lens,
                             const int32_t* src_pending, hipStream_t st) {
  hipLaunchKernelGGL(copy_state_kernel, dim3((B + 63) / 64), dim3(64), 0, st, B, lens, pending, src_lens,
                     src_pending);
  return hipGetLastError();
}

namespace {

// Prompt rows of one prefill forward, per request and in all.  A bf16 cache
// with head_dim 128 takes up to the workspace's rows (the prefill attention
// covers any number of rows per request; the projections then run on the
// wide-row GEMM, every weight tile read once per launch for all rows); other
// caches take kPrefillRows per request (the verify attention's limit).  A
// model setting can lower the rows per request.
void prefill_caps(spade_model md, int* r_cap, int* m_cap) {
  const Dims& D = md->dims;
  const bool tiled = D.kvdt == SPADE_BF16 && D.hd == kAttnHd;
  int r = tiled ? md->ws.Mrows : kPrefillRows;
  if (md->prefill_rows > 0) r = std::min(r, md->prefill_rows);
  *m_cap = tiled ? md->ws.Mrows : md->ws.Mmax;
  *r_cap = std::min(r, *m_cap);
}

}  // namespace

// Requests go through in index order, in ranges [b0, b0 + nb) with R rows
// each: a range starts at the first request with tokens left (R = its
// remaining tokens, up to the caps) and takes in the next requests while all
// nb R rows fit the workspace, every request of the range has R free
// positions in the cache, and at least half the rows are real tokens.  Rows
// depend only on their own token and position, so the cache comes out the
// same as from spade_prefill of each request.
hipError_t launch_prefill_batch(spade_model md, spade_kv kv, int B, const int32_t* tokens, int ld,
                                const int* n_cache, hipStream_t st) {
  const Workspace& W = md->ws;
  for (int b0 = 0; b0 < B; b0 += 64) {
    PrefillCounts c{};
    const int nb = std::min(64, B - b0);
    for (int i = 0; i < nb; ++i) c.n[i] = n_cache[b0 + i];
    hipLaunchKernelGGL(prefill_counts_kernel, dim3(1), dim3(64), 0, st, c, b0, nb, W.prefill_cnt, kv->lens,
                       W.prefill_base);
  }
  int r_cap, m_cap;
  prefill_caps(md, &r_cap, &m_cap);
  std::vector<int> rem(n_cache, n_cache + B);
  hipError_t e = hipGetLastError();
  int b0 = 0;
  while (e == hipSuccess) {
    while (b0 < B && rem[b0] == 0) ++b0;
    if (b0 == B) break;
    int R = std::min(rem[b0], r_cap), nb = 1;
    int top = kv->lens_ub[b0];  // the longest cached length of the range
    while (b0 + nb < B) {
      const int c = b0 + nb;
      const int R2 = std::max(R, std::min(rem[c], r_cap));
      const int top2 = std::max(top, kv->lens_ub[c]);
      if ((long)(nb + 1) * R2 > m_cap || top2 + R2 > kv->max_len) break;
      long real2 = 0;
      for (int b = b0; b <= c; ++b) real2 += std::min(rem[b], R2);
      if (2 * real2 < (long)(nb + 1) * R2) break;
      R = R2;
      top = top2;
      ++nb;
    }
    hipLaunchKernelGGL(prefill_gather_kernel, dim3((nb * R + 255) / 256), dim3(256), 0, st, tokens, ld,
                       W.prefill_cnt, W.prefill_base, kv->lens, b0, nb, R, W.prefill_tok);
    ForwardCall fc{};
    fc.b0 = b0;
    fc.nb = nb;
    fc.R = R;
    fc.tokens = W.prefill_tok;
    fc.want_logits = false;
    e = launch_forward(md, kv, fc, st);
    if (e == hipSuccess) {
      hipLaunchKernelGGL(prefill_advance_kernel, dim3((nb + 63) / 64), dim3(64), 0, st, b0, nb, R, W.prefill_cnt,
                         W.prefill_base, kv->lens);
      e = hipGetLastError();
    }
    // the host bound of lens follows the device lengths (the next forward
    // sizes its attention grid from it)
    for (int b = b0; b < b0 + nb; ++b) {
      const int t = std::min(rem[b], R);
      rem[b] -= t;
      kv->lens_ub[b] += t;
    }
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(prefill_pending_kernel, dim3((B + 63) / 64), dim3(64), 0, st, B, tokens, ld, W.prefill_cnt,
                     kv->pending);
  return hipGetLastError();
}

// One request: forwards of up to the caps' rows over its prompt, then its
// last token becomes pending.
hipError_t launch_prefill_one(spade_model md, spade_kv kv, int b, const int32_t* tokens, int n_cache,
                              hipStream_t st) {
  int r_cap, m_cap;
  prefill_caps(md, &r_cap, &m_cap);
  for (int s = 0; s < n_cache;) {
    ForwardCall fc{};
    fc.b0 = b;
    fc.nb = 1;
    fc.R = std::min(r_cap, n_cache - s);
    fc.tokens = tokens + s;
    fc.want_logits = false;
    hipError_t e = launch_forward(md, kv, fc, st);
    if (e == hipSuccess) e = launch_advance(kv, b, fc.R, nullptr, st);
    if (e != hipSuccess) return e;
    kv->lens_ub[b] += fc.R;
    s += fc.R;
  }
  return launch_advance(kv, b, 0, tokens + n_cache, st);
}

hipError_t launch_advance(spade_kv kv, int b, int count, const int32_t* pending_src, hipStream_t st) {
  hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(64), 0, st, b, count, kv->lens, kv->pending, pending_src);
  return hipGetLastError();
}

}  // namespace spade
