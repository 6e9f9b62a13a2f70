// HIP kernels of the speculative-verify path for gfx950 (MI355X).
//
// One verify pass of SPADE's cloud verifier (Algorithm 1, Cloud step): the
// gamma+1 rows [pending, d_1 .. d_gamma] of every request go through the
// decoder in one pass (Sec. III-A), the LM-head logits give the softmax rows,
// and the accept/reject chain with its correction draw (Sec. III-C) runs on
// the device.
//
// Kernels
//   embed_kernel      x = E[token]; first GEMM operand and RMS partials
//   gemm_kernel       Y = X W^T for skinny X (<= 32 rows), bf16 or f32 weights
//                     streamed from a tiled arena, MFMA 16x16x32 bf16 (the fp32
//                     activations split into three bf16 terms) or 16x16x4 f32,
//                     with fused epilogues: RMSNorm scale + RoPE + KV append
//                     (QKV), residual add + next RMS partials (O, down),
//                     SiLU-gate (gate/up), logits (LM head)
//   attn_kernel       multi-query causal attention of the gamma+1 rows over
//                     the cache, split over key chunks; the last chunk to
//                     finish merges the partials in a fixed order
//   accept_kernel     per request: vocabulary-wide max / log-sum-exp / argmax
//                     per row, the accept chain, the correction draw
//   commit_kernel     lens += n + 1, pending = correction
//   pack_kernel       row-major weights -> tiled arena
#include "spade_internal.h"

#include <float.h>
#include <math.h>

#include <algorithm>

namespace spade {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;

constexpr int kS = 3;  // bf16 terms per fp32 activation (hi, mid, lo)

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Store v as the next GEMM's operand: three bf16 terms (bf16 weights) or the
// float itself (fp32 weights).
template <bool ABF16>
__device__ __forceinline__ void store_act(void* base, size_t split, size_t idx, float v) {
  if constexpr (ABF16) {
    uint16_t* p = (uint16_t*)base;
    float r = v;
#pragma unroll
    for (int s = 0; s < kS; ++s) {
      const uint16_t h = f2bf(r);
      p[s * split + idx] = h;
      r -= bf2f(h);
    }
  } else {
    ((float*)base)[idx] = v;
  }
}

__device__ __forceinline__ void flag_error(uint32_t* err, uint32_t bits) {
  if (err) atomicOr(err, bits);
}

// ---------------------------------------------------------------------------
// Embedding: x_0 = E[token] (Sec. III-A), written with the split operand of
// the first QKV GEMM (x * g_attn of layer 0) and per-16-column sums of x^2.
// ---------------------------------------------------------------------------
struct EmbedParams {
  const void* E;
  const float* g;
  const int32_t* tokens;   // prefill ids [R] or NULL
  const int32_t* drafts;   // [nb][R-1]
  const int32_t* pending;  // global [Bmax]
  int b0, R, d, V;
  float* x;
  void* act;
  size_t act_split;
  float* ssq;
  uint32_t* err;
};

template <bool WBF16>
__global__ void __launch_bounds__(256) embed_kernel(EmbedParams p) {
  const int m = blockIdx.x;
  const int bl = m / p.R, i = m % p.R;
  int t;
  if (p.tokens) t = p.tokens[i];
  else t = (i == 0) ? p.pending[p.b0 + bl] : p.drafts[bl * (p.R - 1) + i - 1];
  if (t < 0 || t >= p.V) {
    if (threadIdx.x == 0) flag_error(p.err, SPADE_DERR_TOKEN);
    t = t < 0 ? 0 : p.V - 1;
  }
  const int npan = p.d / 16;
  for (int pn = threadIdx.x; pn < npan; pn += blockDim.x) {
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int n = pn * 16 + e;
      float v;
      if constexpr (WBF16) v = bf2f(((const uint16_t*)p.E)[(size_t)t * p.d + n]);
      else v = ((const float*)p.E)[(size_t)t * p.d + n];
      p.x[(size_t)m * p.d + n] = v;
      ss += v * v;
      store_act<WBF16>(p.act, p.act_split, (size_t)m * p.d + n, v * p.g[n]);
    }
    p.ssq[(size_t)m * npan + pn] = ss;
  }
}

// ---------------------------------------------------------------------------
// Skinny GEMM with fused epilogues.
//
// Work unit = P weight panels (16 rows each) x all of K; one workgroup per
// unit, NW waves splitting K into contiguous k-block ranges.  A wave streams
// its k-blocks (8 KB per panel) with 16-byte loads: in the arena, slice j of
// a k-block holds for lane l the 8 bf16 (4 f32) weights of row l%16 at
// k = kb*256 + 32j + 8(l/16) (f32: kb*128 + 16j + 4(l/16)), exactly the B
// operand of MFMA j, so every load instruction reads 1 KB contiguous.  The
// A operand (activations, <= 32 rows) is read from L2 with the same k map.
// Partial sums of the waves are reduced in LDS in wave order.
// ---------------------------------------------------------------------------
struct GemmParams {
  const uint8_t* w;
  int NKB;
  int M, m0;
  const void* act;
  size_t act_split;
  int act_stride;
  // row scale 1/rms from partials (ssq_in == NULL: scale 1)
  const float* ssq_in;
  int n_ssq;
  float inv_din, eps;
  int R, b0;
  const int32_t* lens;
  // QKV
  float* q_out;
  void* kc;
  void* vc;
  int H, hd, d, max_len, kv_bf16;
  const float* rope;
  // O / DOWN
  float* x;
  void* act_out;
  size_t act_out_split;
  int act_out_stride;
  const float* g_next;
  float* ssq_out;
  int n_ssq_out;
  // GU
  int F;
  // LM
  float* logits;
  int V;
  uint32_t* err;
};

template <bool WBF16, int P, int NW, int MT, int KIND>
__global__ void __launch_bounds__(NW * 64) gemm_kernel(GemmParams a) {
  const int u = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  __shared__ float red[NW][P][MT][4][64];
  __shared__ float rinv_s[MT * 16];

  if (tid < MT * 16) {
    float r = 1.f;
    if (a.ssq_in != nullptr && tid < a.M) {
      const float* sp = a.ssq_in + (size_t)(a.m0 + tid) * a.n_ssq;
      float s = 0.f;
      for (int i = 0; i < a.n_ssq; ++i) s += sp[i];
      r = 1.0f / sqrtf(s * a.inv_din + a.eps);
    }
    rinv_s[tid] = r;
  }

  floatx4 acc[P][MT];
#pragma unroll
  for (int pp = 0; pp < P; ++pp)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[pp][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int NKB = a.NKB;
  const int kb0 = (NKB * wave) / NW, kb1 = (NKB * (wave + 1)) / NW;
  const uint8_t* wp = a.w + (size_t)u * NKB * P * kTileBytes + lane * 16;
  const int arow = lane & 15, ag = lane >> 4;

  for (int kb = kb0; kb < kb1; ++kb) {
    uint4 wv[P][8];
#pragma unroll
    for (int pp = 0; pp < P; ++pp)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        wv[pp][j] = *(const uint4*)(wp + ((size_t)kb * P + pp) * kTileBytes + j * 1024);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int row = mt * 16 + arow;
      const bool ok = row < a.M;
      if constexpr (WBF16) {
        const uint16_t* ap = (const uint16_t*)a.act + (size_t)(a.m0 + row) * a.act_stride + kb * 256 + ag * 8;
        uint4 av[kS][8];
#pragma unroll
        for (int s = 0; s < kS; ++s)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            av[s][j] = ok ? *(const uint4*)(ap + s * a.act_split + j * 32) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int pp = 0; pp < P; ++pp)
#pragma unroll
            for (int s = kS - 1; s >= 0; --s)
              acc[pp][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, av[s][j]), __builtin_bit_cast(bf16x8, wv[pp][j]),
                  acc[pp][mt], 0, 0, 0);
      } else {
        const float* ap = (const float*)a.act + (size_t)(a.m0 + row) * a.act_stride + kb * 128 + ag * 4;
        float4 av[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) av[j] = ok ? *(const float4*)(ap + j * 16) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int pp = 0; pp < P; ++pp) {
            const float4 w4 = __builtin_bit_cast(float4, wv[pp][j]);
            acc[pp][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j].x, w4.x, acc[pp][mt], 0, 0, 0);
            acc[pp][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j].y, w4.y, acc[pp][mt], 0, 0, 0);
            acc[pp][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j].z, w4.z, acc[pp][mt], 0, 0, 0);
            acc[pp][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j].w, w4.w, acc[pp][mt], 0, 0, 0);
          }
      }
    }
  }

#pragma unroll
  for (int pp = 0; pp < P; ++pp)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][pp][mt][r][lane] = acc[pp][mt][r];
  __syncthreads();

  // Epilogue: thread t <-> accumulator element (mt, r, lane) of every panel;
  // D[i][j] of a 16x16 MFMA sits in lane j + 16*(i/4), register i%4, so the
  // element is row m = mt*16 + 4*(lane/16) + r, panel column n = lane%16.
  if (tid >= MT * 256) return;
  const int emt = tid >> 8, er = (tid >> 6) & 3, eln = tid & 63;
  const int ml = emt * 16 + 4 * (eln >> 4) + er;  // row within this launch
  const int n = eln & 15;
  float val[P];
#pragma unroll
  for (int pp = 0; pp < P; ++pp) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[w][pp][emt][er][eln];
    val[pp] = s;
  }
  const bool rowok = ml < a.M;
  const int m = a.m0 + ml;  // row within the forward call
  const float rinv = rinv_s[ml];

  if constexpr (KIND == GEMM_QKV) {
    if (!rowok) return;
    const int upsec = a.d / 32, uph = a.hd / 32;
    const int sec = u / upsec, rem = u % upsec;
    const int h = rem / uph, wpan = rem % uph;
    const int f0 = wpan * 16 + n, f1 = f0 + a.hd / 2;
    float v0 = val[0] * rinv, v1 = val[1] * rinv;
    const int bl = m / a.R, i = m % a.R;
    const int bg = a.b0 + bl;
    const int pos = a.lens[bg] + i;
    if (sec < 2) {
      const float* cs = a.rope + ((size_t)pos * (a.hd / 2) + f0) * 2;
      const float c = cs[0], sn = cs[1];
      const float o0 = v0 * c - v1 * sn, o1 = v0 * sn + v1 * c;
      v0 = o0;
      v1 = o1;
    }
    if (sec == 0) {
      a.q_out[(size_t)m * a.d + h * a.hd + f0] = v0;
      a.q_out[(size_t)m * a.d + h * a.hd + f1] = v1;
    } else {
      void* cache = sec == 1 ? a.kc : a.vc;
      const size_t off = (((size_t)bg * a.H + h) * a.max_len + pos) * a.hd;
      if (a.kv_bf16) {
        ((uint16_t*)cache)[off + f0] = f2bf(v0);
        ((uint16_t*)cache)[off + f1] = f2bf(v1);
      } else {
        ((float*)cache)[off + f0] = v0;
        ((float*)cache)[off + f1] = v1;
      }
    }
  } else if constexpr (KIND == GEMM_O || KIND == GEMM_DOWN) {
    const int col = u * 16 + n;
    float xv = 0.f;
    if (rowok) {
      xv = a.x[(size_t)m * a.d + col] + val[0];
      a.x[(size_t)m * a.d + col] = xv;
      store_act<WBF16>(a.act_out, a.act_out_split, (size_t)m * a.act_out_stride + col, xv * a.g_next[col]);
    }
    float sq = xv * xv;
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) sq += __shfl_xor(sq, off);
    if (rowok && n == 0) a.ssq_out[(size_t)m * a.n_ssq_out + u] = sq;
  } else if constexpr (KIND == GEMM_GU) {
    if (!rowok) return;
    const int col = u * 16 + n;
    const float gv = val[0] * rinv, uv = val[1] * rinv;
    const float act = gv / (1.0f + expf(-gv)) * uv;
    store_act<WBF16>(a.act_out, a.act_out_split, (size_t)m * a.act_out_stride + col, act);
  } else {  // GEMM_LM
    const int col = u * 16 + n;
    if (!rowok || col >= a.V) return;
    const float lg = val[0] * rinv;
    if (lg != lg) flag_error(a.err, SPADE_DERR_NAN);
    a.logits[(size_t)m * a.V + col] = lg;
  }
}

// ---------------------------------------------------------------------------
// Verify attention.  Workgroup (chunk c, head h, request b): the R query rows
// of the request against keys [c*CK, min((c+1)*CK, L_b + R)), key j visible
// to row i iff j <= L_b + i (causal inside the appended block).  Sixteen
// lanes share a key (HD/16 features each), four keys per wave step.  Each
// chunk writes (max, sum, unnormalised output) per row; the workgroup that
// finishes last for (b, h) merges the chunks in chunk order and writes the
// O-projection operand.
// ---------------------------------------------------------------------------
struct AttnParams {
  const float* q;
  const void* kc;
  const void* vc;
  const int32_t* lens;
  int b0, R, H, d, max_len;
  int CK, NC;
  float scale;
  float* part_o;
  float* part_ml;
  uint32_t* cnt;
  int Rmax;
  void* act_out;
  size_t act_split;
};

constexpr int kAttnMaxCK = 256;

template <int HD, bool KVBF16>
__device__ __forceinline__ void load_kv(const void* base, size_t off, float* out) {
  constexpr int DPL = HD / 16;
  if constexpr (KVBF16) {
    const uint16_t* p = (const uint16_t*)base + off;
    if constexpr (DPL == 8) {
      const uint4 v = *(const uint4*)p;
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        out[2 * e] = __uint_as_float(w[e] << 16);
        out[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int e = 0; e < DPL; ++e) out[e] = bf2f(p[e]);
    }
  } else {
    const float* p = (const float*)base + off;
#pragma unroll
    for (int e = 0; e < DPL; e += 4) {
      const float4 v = *(const float4*)(p + e);
      out[e] = v.x;
      out[e + 1] = v.y;
      out[e + 2] = v.z;
      out[e + 3] = v.w;
    }
  }
}

template <int HD, bool KVBF16, bool ABF16>
__global__ void __launch_bounds__(256) attn_kernel(AttnParams p) {
  constexpr int DPL = HD / 16;
  const int c = blockIdx.x, h = blockIdx.y, bl = blockIdx.z;
  const int bg = p.b0 + bl;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kg = lane >> 4, dg = lane & 15;
  const int R = p.R;
  const int L = p.lens[bg];
  const int nkeys = L + R;
  const int k_lo = c * p.CK;
  const int k_hi = min(k_lo + p.CK, nkeys);

  __shared__ float s_lds[kMaxR][kAttnMaxCK];
  __shared__ float o_lds[4][kMaxR][HD];
  __shared__ float m_lds[kMaxR], l_lds[kMaxR];
  __shared__ int last_s;

  const size_t bh = (size_t)bl * p.H + h;
  float* po = p.part_o + ((bh * p.NC + c) * p.Rmax) * HD;
  float* pml = p.part_ml + ((bh * p.NC + c) * p.Rmax) * 2;
  const size_t kvbase = ((size_t)bg * p.H + h) * p.max_len * HD;

  if (k_lo < k_hi) {
    // scores
    float qr[kMaxR][DPL];
#pragma unroll
    for (int r = 0; r < kMaxR; ++r)
#pragma unroll
      for (int e = 0; e < DPL; ++e)
        qr[r][e] = r < R ? p.q[(size_t)(bl * R + r) * p.d + h * HD + dg * DPL + e] : 0.f;
    for (int kb = k_lo + 4 * wave; kb < k_hi; kb += 16) {
      const int k = kb + kg;
      float kv[DPL];
      if (k < k_hi) load_kv<HD, KVBF16>(p.kc, kvbase + (size_t)k * HD + dg * DPL, kv);
      else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) kv[e] = 0.f;
      }
      float dot[kMaxR];
#pragma unroll
      for (int r = 0; r < kMaxR; ++r) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) s += qr[r][e] * kv[e];
        dot[r] = s;
      }
#pragma unroll
      for (int r = 0; r < kMaxR; ++r) {
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) dot[r] += __shfl_xor(dot[r], off);
      }
      float mine = 0.f;
#pragma unroll
      for (int r = 0; r < kMaxR; ++r)
        if (r == dg) mine = dot[r];
      if (k < k_hi && dg < R) s_lds[dg][k - k_lo] = (k <= L + dg) ? mine * p.scale : -INFINITY;
    }
    __syncthreads();
    // chunk softmax, one wave per row
    const int nk = k_hi - k_lo;
    for (int r = wave; r < R; r += 4) {
      float mx = -INFINITY;
      for (int j = lane; j < nk; j += 64) mx = fmaxf(mx, s_lds[r][j]);
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
      float sum = 0.f;
      for (int j = lane; j < nk; j += 64) {
        const float e = (mx == -INFINITY) ? 0.f : expf(s_lds[r][j] - mx);
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
    // P V
    float acc[kMaxR][DPL];
#pragma unroll
    for (int r = 0; r < kMaxR; ++r)
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[r][e] = 0.f;
    for (int kb = k_lo + 4 * wave; kb < k_hi; kb += 16) {
      const int k = kb + kg;
      if (k < k_hi) {
        float vv[DPL];
        load_kv<HD, KVBF16>(p.vc, kvbase + (size_t)k * HD + dg * DPL, vv);
#pragma unroll
        for (int r = 0; r < kMaxR; ++r) {
          if (r < R) {
            const float pr = s_lds[r][k - k_lo];
#pragma unroll
            for (int e = 0; e < DPL; ++e) acc[r][e] += pr * vv[e];
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < kMaxR; ++r)
#pragma unroll
      for (int e = 0; e < DPL; ++e) {
        float v = acc[r][e];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        acc[r][e] = v;
      }
    if (kg == 0) {
#pragma unroll
      for (int r = 0; r < kMaxR; ++r)
        if (r < R)
#pragma unroll
          for (int e = 0; e < DPL; ++e) o_lds[wave][r][dg * DPL + e] = acc[r][e];
    }
    __syncthreads();
    for (int idx = tid; idx < R * HD; idx += 256) {
      const int r = idx / HD, dd = idx % HD;
      po[r * HD + dd] = o_lds[0][r][dd] + o_lds[1][r][dd] + o_lds[2][r][dd] + o_lds[3][r][dd];
    }
    if (tid < R) {
      pml[tid * 2] = m_lds[tid];
      pml[tid * 2 + 1] = l_lds[tid];
    }
  } else {
    if (tid < R) {
      pml[tid * 2] = -INFINITY;
      pml[tid * 2 + 1] = 0.f;
    }
  }

  // the last chunk of (b, h) to arrive merges
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = atomicAdd(&p.cnt[bh], 1u);
    last_s = (old == (uint32_t)(p.NC - 1));
  }
  __syncthreads();
  if (!last_s) return;
  __threadfence();
  const float* po0 = p.part_o + (bh * p.NC * p.Rmax) * HD;
  const float* pml0 = p.part_ml + (bh * p.NC * p.Rmax) * 2;
  for (int idx = tid; idx < R * HD; idx += 256) {
    const int r = idx / HD, dd = idx % HD;
    float M = -INFINITY;
    for (int cc = 0; cc < p.NC; ++cc) M = fmaxf(M, __builtin_nontemporal_load(pml0 + ((size_t)cc * p.Rmax + r) * 2));
    float Ls = 0.f, O = 0.f;
    for (int cc = 0; cc < p.NC; ++cc) {
      const float mc = __builtin_nontemporal_load(pml0 + ((size_t)cc * p.Rmax + r) * 2);
      if (mc == -INFINITY) continue;
      const float sc = expf(mc - M);
      Ls += __builtin_nontemporal_load(pml0 + ((size_t)cc * p.Rmax + r) * 2 + 1) * sc;
      O += __builtin_nontemporal_load(po0 + ((size_t)cc * p.Rmax + r) * HD + dd) * sc;
    }
    const int m = bl * R + r;
    store_act<ABF16>(p.act_out, p.act_split, (size_t)m * p.d + h * HD + dd, O / Ls);
  }
  if (tid == 0) p.cnt[bh] = 0u;
}

// ---------------------------------------------------------------------------
// Accept / reject and the correction draw, one workgroup per request
// (Sec. III-C; Algorithm 1, the verify / accept / sample / correct steps).
// ---------------------------------------------------------------------------
struct AcceptParams {
  const float* logits;
  int V, gamma, R;
  const int32_t* drafts;
  const float* q;
  const float* u;
  const uint8_t* mode;
  float inv_T;
  int32_t* n_out;
  int32_t* corr_out;
  uint32_t* err;
};

// SplitMix64 output v (0-based) of the stream seeded with `seed`.
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t v) {
  uint64_t z = seed + (v + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ float gumbel_at(uint64_t seed, int v) {
  const uint64_t x = splitmix64_at(seed, (uint64_t)v);
  const float U = ((float)(uint32_t)(x >> 41) + 0.5f) * 0x1p-23f;
  return -logf(-logf(U));
}

// (max, sum exp(z - max), argmax) merge; ties keep the lower id.
struct RowStat {
  float m, s;
  int a;
};

__device__ __forceinline__ RowStat merge_stat(RowStat x, RowStat y) {
  if (y.m > x.m || (y.m == x.m && y.a < x.a && y.m != -INFINITY)) {
    const RowStat t = x;
    x = y;
    y = t;
  }
  // x has the larger max (or equal max with lower id)
  RowStat o;
  o.m = x.m;
  o.a = x.a;
  o.s = x.s + ((y.m == -INFINITY) ? 0.f : y.s * expf(y.m - x.m));
  return o;
}

__device__ __forceinline__ RowStat wave_merge(RowStat st) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    RowStat o;
    o.m = __shfl_xor(st.m, off);
    o.s = __shfl_xor(st.s, off);
    o.a = __shfl_xor(st.a, off);
    // combine in lane order so every lane reaches the same result
    const bool lower = (threadIdx.x & off) == 0;
    st = lower ? merge_stat(st, o) : merge_stat(o, st);
  }
  return st;
}

struct Best {
  float s;
  int a;
};

__device__ __forceinline__ Best better(Best x, Best y) {
  if (y.s > x.s || (y.s == x.s && y.a < x.a)) return y;
  return x;
}

__global__ void __launch_bounds__(256) accept_kernel(AcceptParams p) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int R = p.R, V = p.V, G = p.gamma;
  __shared__ float rmax[kMaxR + 1], rlse[kMaxR + 1];
  __shared__ int rarg[kMaxR + 1];
  __shared__ RowStat part[4];
  __shared__ Best bpart[4];
  __shared__ int n_s;

  bool sample = p.mode[b] == SPADE_SAMPLE;
  if (sample && (p.u == nullptr || (G > 0 && p.q == nullptr))) {
    if (tid == 0) flag_error(p.err, SPADE_DERR_NOQ);
    sample = false;
  }
  const float invT = sample ? p.inv_T : 1.0f;
  const float* lg = p.logits + (size_t)b * R * V;

  // row statistics over the vocabulary
  for (int r = 0; r < R; ++r) {
    RowStat st{-INFINITY, 0.f, 0x7fffffff};
    for (int v = tid; v < V; v += 256) {
      const float z = lg[(size_t)r * V + v] * invT;
      if (z != z) continue;
      RowStat one{z, 1.f, v};
      st = merge_stat(st, one);
    }
    st = wave_merge(st);
    if (lane == 0) part[wave] = st;
    __syncthreads();
    if (tid == 0) {
      RowStat t = part[0];
      for (int w = 1; w < 4; ++w) t = merge_stat(t, part[w]);
      rmax[r] = t.m;
      rlse[r] = t.m + logf(t.s);
      rarg[r] = t.a;
    }
    __syncthreads();
  }

  if (tid == 0) {
    int n = G;
    for (int i = 0; i < G; ++i) {
      int x = p.drafts[(size_t)b * G + i];
      if (x < 0 || x >= V) {
        flag_error(p.err, SPADE_DERR_TOKEN);
        x = x < 0 ? 0 : V - 1;
      }
      bool ok;
      if (!sample) {
        ok = (x == rarg[i]);
      } else {
        const float px = expf(lg[(size_t)i * V + x] * invT - rlse[i]);
        const float qx = p.q[((size_t)b * G + i) * V + x];
        ok = p.u[(size_t)b * (G + 1) + i] * qx < px;
      }
      if (!ok) {
        n = i;
        break;
      }
    }
    n_s = n;
  }
  __syncthreads();
  const int n = n_s;
  int corr = 0;
  if (!sample) {
    corr = rarg[n];
  } else {
    const uint64_t seed = (uint64_t)__float_as_uint(p.u[(size_t)b * (G + 1) + G]);
    const float* row = lg + (size_t)n * V;
    const bool residual = n < G;
    const float* qrow = residual ? p.q + ((size_t)b * G + n) * V : nullptr;
    const float lse = rlse[n];
    for (int pass = 0; pass < 2; ++pass) {
      const bool use_res = residual && pass == 0;
      Best bst{-INFINITY, 0x7fffffff};
      for (int v = tid; v < V; v += 256) {
        const float z = row[v] * invT;
        float sc;
        if (use_res) {
          const float w = expf(z - lse) - qrow[v];
          sc = w > 0.f ? logf(w) + gumbel_at(seed, v) : -INFINITY;
        } else {
          sc = z + gumbel_at(seed, v);
        }
        if (sc != sc) continue;
        bst = better(bst, Best{sc, v});
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        Best o{__shfl_xor(bst.s, off), __shfl_xor(bst.a, off)};
        bst = better(bst, o);
      }
      if (lane == 0) bpart[wave] = bst;
      __syncthreads();
      Best t = bpart[0];
      for (int w = 1; w < 4; ++w) t = better(t, bpart[w]);
      __syncthreads();
      if (t.s != -INFINITY || !use_res) {
        corr = t.a;
        break;
      }
      if (tid == 0) flag_error(p.err, SPADE_DERR_RESIDUAL);
    }
  }
  if (tid == 0) {
    p.n_out[b] = n;
    p.corr_out[b] = corr;
  }
}

// ---------------------------------------------------------------------------
// Small kernels: commit, lens advance, inverse temperatures, packing.
// ---------------------------------------------------------------------------
__global__ void commit_kernel(int B, int32_t* lens, int32_t* pending, const int32_t* n, const int32_t* corr) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) {
    lens[b] += n[b] + 1;
    pending[b] = corr[b];
  }
}

__global__ void advance_kernel(int b, int count, int32_t* lens, int32_t* pending, const int32_t* src) {
  if (threadIdx.x == 0) {
    lens[b] += count;
    if (src) pending[b] = *src;
  }
}

struct PackParams {
  const uint8_t* src;
  uint8_t* dst;
  int kind, wbf16;
  int N_src, row_off, K, NKB, KB, P, n_units, N_logical, pad_from;
  int d, hd, F;
};

__global__ void pack_kernel(PackParams p) {
  const size_t chunk = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)p.n_units * p.NKB * p.P * 512;  // 16-byte chunks
  if (chunk >= total) return;
  const int lane = (int)(chunk & 63);
  const int j = (int)((chunk >> 6) & 7);
  size_t t = chunk >> 9;
  const int pp = (int)(t % p.P);
  t /= p.P;
  const int kb = (int)(t % p.NKB);
  const int u = (int)(t / p.NKB);
  const int panel = unit_panel(p.kind, u, pp, p.d, p.hd, p.F);
  const int row = panel * 16 + (lane & 15);
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

template <bool WBF16, int P, int KIND>
hipError_t launch_gemm_kind(const GemmParams& gp, int units, int mt, hipStream_t st) {
  constexpr int NW = 8;
  if (mt == 1)
    hipLaunchKernelGGL((gemm_kernel<WBF16, P, NW, 1, KIND>), dim3(units), dim3(NW * 64), 0, st, gp);
  else
    hipLaunchKernelGGL((gemm_kernel<WBF16, P, NW, 2, KIND>), dim3(units), dim3(NW * 64), 0, st, gp);
  return hipGetLastError();
}

template <bool WBF16>
hipError_t launch_gemm(int kind, const GemmParams& gp, int units, int mt, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_gemm_kind<WBF16, 2, GEMM_QKV>(gp, units, mt, st);
    case GEMM_O: return launch_gemm_kind<WBF16, 1, GEMM_O>(gp, units, mt, st);
    case GEMM_GU: return launch_gemm_kind<WBF16, 2, GEMM_GU>(gp, units, mt, st);
    case GEMM_DOWN: return launch_gemm_kind<WBF16, 1, GEMM_DOWN>(gp, units, mt, st);
    default: return launch_gemm_kind<WBF16, 1, GEMM_LM>(gp, units, mt, st);
  }
}

template <int HD>
hipError_t launch_attn_hd(const AttnParams& ap, bool kvbf16, bool abf16, dim3 grid, hipStream_t st) {
  if (kvbf16 && abf16) hipLaunchKernelGGL((attn_kernel<HD, true, true>), grid, dim3(256), 0, st, ap);
  else if (kvbf16) hipLaunchKernelGGL((attn_kernel<HD, true, false>), grid, dim3(256), 0, st, ap);
  else if (abf16) hipLaunchKernelGGL((attn_kernel<HD, false, true>), grid, dim3(256), 0, st, ap);
  else hipLaunchKernelGGL((attn_kernel<HD, false, false>), grid, dim3(256), 0, st, ap);
  return hipGetLastError();
}

}  // namespace

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
  if (wb) hipLaunchKernelGGL(embed_kernel<true>, dim3(M), dim3(256), 0, st, ep);
  else hipLaunchKernelGGL(embed_kernel<false>, dim3(M), dim3(256), 0, st, ep);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  const int KBd = kblock_of(D.wdt);
  const size_t kv_layer = (size_t)kv->max_batch * D.H * kv->max_len * D.hd;  // elements
  const size_t kv_elt = D.kvdt == SPADE_BF16 ? 2 : 4;

  // attention chunking: enough workgroups to fill the chip
  int max_keys = 0;
  for (int b = fc.b0; b < fc.b0 + fc.nb; ++b) max_keys = std::max(max_keys, kv->lens_ub[b] + fc.R);
  int CK = kAttnChunkMin;
  while (CK < kAttnMaxCK && (long)fc.nb * D.H * ((max_keys + CK - 1) / CK) > 2048) CK *= 2;
  const int NC = (max_keys + CK - 1) / CK;
  if (NC > W.NCmax) return hipErrorInvalidValue;

  auto gemm = [&](int kind, const uint8_t* wmat, int K, int units, const void* act, size_t act_split,
                  GemmParams base) -> hipError_t {
    for (int m0 = 0; m0 < M; m0 += kMaxRowsPerGemm) {
      GemmParams gp = base;
      gp.w = wmat;
      gp.NKB = K / KBd;
      gp.M = std::min(kMaxRowsPerGemm, M - m0);
      gp.m0 = m0;
      gp.act = act;
      gp.act_split = act_split;
      gp.act_stride = K;
      const int mt = gp.M > 16 ? 2 : 1;
      hipError_t r = wb ? launch_gemm<true>(kind, gp, units, mt, st) : launch_gemm<false>(kind, gp, units, mt, st);
      if (r != hipSuccess) return r;
    }
    return hipSuccess;
  };

  GemmParams common{};
  common.R = fc.R;
  common.b0 = fc.b0;
  common.lens = kv->lens;
  common.inv_din = 1.0f / (float)D.d;
  common.eps = D.eps;
  common.n_ssq = D.d / 16;
  common.H = D.H;
  common.hd = D.hd;
  common.d = D.d;
  common.F = D.F;
  common.max_len = kv->max_len;
  common.kv_bf16 = D.kvdt == SPADE_BF16;
  common.rope = W.rope;
  common.x = W.x;
  common.V = D.V;
  common.err = W.err;

  for (int l = 0; l < D.L; ++l) {
    const uint8_t* lb = md->weights + (size_t)l * md->lay.layer_bytes;
    // QKV + RoPE + KV append
    GemmParams g = common;
    g.ssq_in = W.ssq;
    g.q_out = W.q;
    g.kc = kv->k + (size_t)l * kv_layer * kv_elt;
    g.vc = kv->v + (size_t)l * kv_layer * kv_elt;
    if ((e = gemm(GEMM_QKV, lb + md->lay.qkv, D.d, 3 * D.d / 32, W.act_n, W.act_split, g)) != hipSuccess) return e;
    // attention
    AttnParams ap{};
    ap.q = W.q;
    ap.kc = g.kc;
    ap.vc = g.vc;
    ap.lens = kv->lens;
    ap.b0 = fc.b0;
    ap.R = fc.R;
    ap.H = D.H;
    ap.d = D.d;
    ap.max_len = kv->max_len;
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
    if (D.hd == 64) e = launch_attn_hd<64>(ap, kvb, wb, agrid, st);
    else e = launch_attn_hd<128>(ap, kvb, wb, agrid, st);
    if (e != hipSuccess) return e;
    // O projection + residual; operand of gate/up = x * g_ffn
    g = common;
    g.act_out = W.act_n;
    g.act_out_split = W.act_split;
    g.act_out_stride = D.d;
    g.g_next = (const float*)(lb + md->lay.g_ffn);
    g.ssq_out = W.ssq;
    g.n_ssq_out = D.d / 16;
    if ((e = gemm(GEMM_O, lb + md->lay.o, D.d, D.d / 16, W.act_o, W.act_split, g)) != hipSuccess) return e;
    // gate/up + SiLU
    g = common;
    g.ssq_in = W.ssq;
    g.act_out = W.act_f;
    g.act_out_split = W.actf_split;
    g.act_out_stride = D.F;
    if ((e = gemm(GEMM_GU, lb + md->lay.gu, D.d, D.F / 16, W.act_n, W.act_split, g)) != hipSuccess) return e;
    // down + residual; operand of the next layer (or the LM head)
    g = common;
    g.act_out = W.act_n;
    g.act_out_split = W.act_split;
    g.act_out_stride = D.d;
    g.g_next = (l + 1 < D.L) ? (const float*)(md->weights + (size_t)(l + 1) * md->lay.layer_bytes + md->lay.g_attn)
                             : (const float*)(md->weights + md->lay.g_final);
    g.ssq_out = W.ssq;
    g.n_ssq_out = D.d / 16;
    if ((e = gemm(GEMM_DOWN, lb + md->lay.down, D.F, D.d / 16, W.act_f, W.actf_split, g)) != hipSuccess) return e;
  }
  if (fc.want_logits) {
    GemmParams g = common;
    g.ssq_in = W.ssq;
    g.logits = fc.logits_out;
    if ((e = gemm(GEMM_LM, md->weights + md->lay.lm, D.d, D.Vpad / 16, W.act_n, W.act_split, g)) != hipSuccess)
      return e;
  }
  return hipSuccess;
}

hipError_t launch_accept(spade_model md, int B, int gamma, int V, const float* logits, bool /*have_stats*/,
                         const int32_t* drafts, const float* q, const float* u, const uint8_t* mode,
                         float temperature, int32_t* n_out, int32_t* corr_out, hipStream_t st) {
  AcceptParams p{};
  p.logits = logits;
  p.V = V;
  p.gamma = gamma;
  p.R = gamma + 1;
  p.drafts = drafts;
  p.q = q;
  p.u = u;
  p.mode = mode;
  p.inv_T = temperature > 0.f ? 1.0f / temperature : 1.0f;
  p.n_out = n_out;
  p.corr_out = corr_out;
  p.err = md->ws.err;
  hipLaunchKernelGGL(accept_kernel, dim3(B), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_pack(spade_model md, int kind, int layer, const void* src, hipStream_t st) {
  const Dims& D = md->dims;
  const bool wb = D.wdt == SPADE_BF16;
  const size_t elt = wb ? 2 : 4;
  const uint8_t* lb = md->weights + (size_t)layer * md->lay.layer_bytes;
  size_t bytes = 0;
  uint8_t* dst = nullptr;
  PackParams pp{};
  pp.src = (const uint8_t*)src;
  pp.wbf16 = wb;
  pp.KB = kblock_of(D.wdt);
  pp.d = D.d;
  pp.hd = D.hd;
  pp.F = D.F;
  switch (kind) {
    case SPADE_WQ: case SPADE_WK: case SPADE_WV:
      pp.kind = GEMM_QKV; pp.K = D.d; pp.N_src = D.d; pp.row_off = (kind - SPADE_WQ) * D.d;
      pp.N_logical = 3 * D.d; pp.n_units = 3 * D.d / 32; dst = (uint8_t*)lb + md->lay.qkv; break;
    case SPADE_WO:
      pp.kind = GEMM_O; pp.K = D.d; pp.N_src = D.d; pp.row_off = 0; pp.N_logical = D.d;
      pp.n_units = D.d / 16; dst = (uint8_t*)lb + md->lay.o; break;
    case SPADE_WGATE: case SPADE_WUP:
      pp.kind = GEMM_GU; pp.K = D.d; pp.N_src = D.F; pp.row_off = (kind - SPADE_WGATE) * D.F;
      pp.N_logical = 2 * D.F; pp.n_units = D.F / 16; dst = (uint8_t*)lb + md->lay.gu; break;
    case SPADE_WDOWN:
      pp.kind = GEMM_DOWN; pp.K = D.F; pp.N_src = D.d; pp.row_off = 0; pp.N_logical = D.d;
      pp.n_units = D.d / 16; dst = (uint8_t*)lb + md->lay.down; break;
    case SPADE_LM_HEAD:
      pp.kind = GEMM_LM; pp.K = D.d; pp.N_src = D.V; pp.row_off = 0; pp.N_logical = D.Vpad;
      pp.n_units = D.Vpad / 16; dst = md->weights + md->lay.lm; break;
    case SPADE_EMBED:
      bytes = (size_t)D.V * D.d * elt;
      return hipMemcpyAsync(md->weights + md->lay.embed, src, bytes, hipMemcpyDeviceToDevice, st);
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
  pp.P = panels_per_unit(pp.kind);
  pp.NKB = pp.K / pp.KB;
  const size_t total = (size_t)pp.n_units * pp.NKB * pp.P * 512;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL(pack_kernel, dim3(blocks), dim3(256), 0, st, pp);
  return hipGetLastError();
}

hipError_t launch_commit(spade_kv kv, int B, const int32_t* n, const int32_t* corr, hipStream_t st) {
  hipLaunchKernelGGL(commit_kernel, dim3((B + 63) / 64), dim3(64), 0, st, B, kv->lens, kv->pending, n, corr);
  return hipGetLastError();
}

hipError_t launch_advance(spade_kv kv, int b, int count, const int32_t* pending_src, hipStream_t st) {
  hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(64), 0, st, b, count, kv->lens, kv->pending, pending_src);
  return hipGetLastError();
}

}  // namespace spade
