// Skinny GEMM engine with fused epilogues.
//
// The arena stores a weight matrix as panels of 16 rows, each panel as its
// k-blocks (256 k for bf16, 128 for f32) of 8 KB.  Slice j of a k-block holds
// for lane l the 8 bf16 (4 f32) weights of panel row l%16 at
// k = kb*256 + 32j + 8(l/16) (f32: kb*128 + 16j + 4(l/16)) -- the B operand of
// MFMA j -- so each wave load instruction reads 1 KB contiguous.
//
// A workgroup of 8 waves takes panels ("units") u = bid, bid + G, ...; each
// wave owns a contiguous k-block range of every unit and walks a stream of
// (unit, k-block) items through a three-deep register pipeline: the weight
// tile of item t+3 is requested while the MFMAs consume item t.  After the
// last item of a unit the wave partials are summed in LDS (in wave order) and
// the unit's epilogue runs.  Activation operands (<= 32 rows) are either
// copied once per launch into LDS (rows <= 16 whose split operand fits: every
// item reads its fragment from there) or fetched from L2 with every item, one
// item ahead.
//
// Every memory access inside the item loop is an unconditional raw-buffer
// instruction whose range check masks absent rows and items (offsets past the
// resource read 0, stores are dropped), and the epilogue's inputs are fetched
// two items ahead.  With no load under a branch the compiler's wait counts
// stay exact, so a wait for item t leaves items t+1 and t+2 in flight.
#pragma once

#include "device_util.h"

namespace spade {

struct GemmParams {
  const uint8_t* w;
  int NKB, n_units;
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
  uint32_t kv_bytes;  // bytes of one layer's K (or V) cache
  int H, hd, d, kv_stride, kv_bf16;
  int Hkv;  // K/V heads (the cache's head count; H for multi-head attention)
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
  float* stats;  // [M][NU][3]: (max, sum exp, argmax) of z = logit (/T) per row and workgroup
  int NU;        // workgroups of the LM-head launch
  float* pstats; // [M][n_units][3]: the same per row and panel (wide-row and split-K LM heads)
  const uint8_t* mode;
  float inv_T;
  int have_q;
  uint32_t* err;
};

constexpr int kGemmWaves = 8;

template <int MT>
struct GemmSmem {
  float red[kGemmWaves][MT][4][64];
  float rinv[MT * 16];
};

// LDS copy of the activation operand: per split, rows 0..M-1, each K elements
// plus 16 bytes of padding (rows start 4 banks apart, so the 16 rows of a
// fragment read hit distinct banks).  MFMA rows past M read row M - 1: their
// outputs are never stored and do not mix with other rows.
inline __host__ __device__ uint32_t gemm_lds_row_bytes(int K, int wbf16) { return (uint32_t)K * (wbf16 ? 2u : 4u) + 16u; }
inline __host__ __device__ uint32_t gemm_lds_a_bytes(int M, int K, int wbf16) {
  return (uint32_t)(wbf16 ? kActSplits : 1) * (uint32_t)M * gemm_lds_row_bytes(K, wbf16);
}
// the LDS copy moves whole 1 KB blocks of a row
inline __host__ __device__ bool gemm_lds_a_ok(int K, int wbf16) { return ((K * (wbf16 ? 2 : 4)) & 1023) == 0; }
constexpr uint32_t kGemmLdsABytes = 144 * 1024;  // largest LDS operand copy

struct EpiIn {
  float a, b;
};

// Epilogue inputs of output (row ml of the launch, column n of unit u) for
// the projection kinds: QKV the RoPE (cos, sin) at position pos, O / down the
// residual x and the next RMSNorm gain.  ok == false reads nothing (zeros).
template <int KIND, bool COH>
__device__ __forceinline__ EpiIn gemm_epi_load(const GemmParams& a, int u, int ml, int n, bool ok, int pos) {
  EpiIn e{0.f, 0.f};
  if constexpr (KIND == GEMM_QKV) {
    const int pph = a.hd >> 4;  // sections start at multiples of pph panels
    const int pair = (u % pph) * 8 + (n & 7);
    const Rsrc rr = make_rsrc(a.rope, 0x7ffffff0u);
    const float2 cs = ld_f32x2<false>(rr, ok ? (uint32_t)((pos * (a.hd >> 1) + pair) * 2) * 4u : kOob);
    e.a = cs.x;
    e.b = cs.y;
  } else if constexpr (KIND == GEMM_O || KIND == GEMM_DOWN) {
    const int col = u * 16 + n;
    const Rsrc rx = make_rsrc(a.x + (size_t)a.m0 * a.d, (uint32_t)((size_t)a.M * a.d * 4));
    const Rsrc rg = make_rsrc(a.g_next, (uint32_t)(a.d * 4));
    e.a = ld_f32<COH>(rx, ok ? (uint32_t)(ml * a.d + col) * 4u : kOob);
    e.b = ld_f32<false>(rg, ok ? (uint32_t)col * 4u : kOob);
  }
  return e;
}

// Epilogue of output (row ml of the launch, column n of unit u) for the
// projection kinds QKV, O, gate/up and down: val is the full dot product,
// rinv the row's 1/rms, e its gemm_epi_load inputs; rok == false stores
// nothing.  D[i][j] of a 16x16 MFMA sits in lane j + 16*(i/4), register i%4,
// so the 16 columns of a row are 16 consecutive lanes: every lane of the wave
// calls it (RoPE and SwiGLU partners are lanes n and n^8, the row's sum of
// squares runs over the 16 lanes).
template <int KIND, bool WBF16, bool COH>
__device__ __forceinline__ void gemm_epilogue(const GemmParams& a, int u, int ml, int n, bool rok, int pos, int bg,
                                              float rinv, float val, const EpiIn& e) {
  constexpr uint32_t ELT = WBF16 ? 2u : 4u;
  constexpr int S = WBF16 ? kActSplits : 1;
  if constexpr (KIND == GEMM_QKV) {
    const int pph = a.hd >> 4;
    int pw;
    const int sec = qkv_section(u, a.d, a.Hkv * a.hd, &pw);
    const int h = pw / pph, wg = pw - h * pph;  // query head (sec 0) or K/V head
    const int pair = wg * 8 + (n & 7);
    const bool hi = n >= 8;
    const int f = pair + (hi ? (a.hd >> 1) : 0);
    float v = val * rinv;
    const float pv = __shfl_xor(v, 8);  // the RoPE partner
    const bool rot = sec < 2;
    const float c = rot ? e.a : 1.f, sn = rot ? e.b : 0.f;
    v = hi ? (pv * sn + v * c) : (v * c - pv * sn);
    const Rsrc rq = make_rsrc(a.q_out + (size_t)a.m0 * a.d, (uint32_t)((size_t)a.M * a.d * 4));
    st_f32<COH>(rq, (rok && sec == 0) ? (uint32_t)(ml * a.d + h * a.hd + f) * 4u : kOob, v);
    // K and V in blocks of kVBlock positions (k_cache_index, v_cache_index;
    // a float32 K cache is [pos][hd])
    const uint32_t head = (uint32_t)(bg * a.Hkv + h) * (uint32_t)a.kv_stride * (uint32_t)a.hd;
    const uint32_t vel = (uint32_t)(a.kv_bf16 ? v_cache_index(f, pos, a.hd) : v_cache_index_f32(f, pos, a.hd));
    const uint32_t kel = (uint32_t)(a.kv_bf16 ? k_cache_index(f, pos, a.hd) : (size_t)pos * a.hd + f);
    const uint32_t elem = head + (sec == 1 ? kel : vel);
    const Rsrc rkv = make_rsrc(sec == 1 ? a.kc : a.vc, a.kv_bytes);
    const bool kok = rok && sec > 0;
    if (a.kv_bf16) st_b16<COH>(rkv, kok ? elem * 2u : kOob, f2bf(v));
    else st_f32<COH>(rkv, kok ? elem * 4u : kOob, v);
  } else if constexpr (KIND == GEMM_O || KIND == GEMM_DOWN) {
    const int col = u * 16 + n;
    const float xv = e.a + val;
    const Rsrc rx = make_rsrc(a.x + (size_t)a.m0 * a.d, (uint32_t)((size_t)a.M * a.d * 4));
    st_f32<COH>(rx, rok ? (uint32_t)(ml * a.d + col) * 4u : kOob, xv);
    const uint32_t split_b = (uint32_t)(a.act_out_split * ELT);
    const Rsrc ro = make_rsrc((const uint8_t*)a.act_out + (size_t)a.m0 * a.act_out_stride * ELT,
                              (uint32_t)((S - 1) * (size_t)split_b + (size_t)a.M * a.act_out_stride * ELT));
    st_act<WBF16, COH>(ro, split_b, (uint32_t)(ml * a.act_out_stride + col), rok, xv * e.b);
    float sq = rok ? xv * xv : 0.f;
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) sq += __shfl_xor(sq, off);
    const Rsrc rs = make_rsrc(a.ssq_out + (size_t)a.m0 * a.n_ssq_out, (uint32_t)((size_t)a.M * a.n_ssq_out * 4));
    st_f32<COH>(rs, (rok && n == 0) ? (uint32_t)(ml * a.n_ssq_out + u) * 4u : kOob, sq);
  } else if constexpr (KIND == GEMM_GU) {
    const float v = val * rinv;
    const float up = __shfl_xor(v, 8);
    const float act = v / (1.0f + expf(-v)) * up;
    const uint32_t split_b = (uint32_t)(a.act_out_split * ELT);
    const Rsrc ro = make_rsrc((const uint8_t*)a.act_out + (size_t)a.m0 * a.act_out_stride * ELT,
                              (uint32_t)((S - 1) * (size_t)split_b + (size_t)a.M * a.act_out_stride * ELT));
    st_act<WBF16, COH>(ro, split_b, (uint32_t)(ml * a.act_out_stride + u * 8 + n), rok && n < 8, act);
  }
}

// LM head: store the logit of (launch row ml, column n of panel u) and return
// the panel's (max, sum exp, argmax) of z = logit (/T for sampling rows) over
// its 16 columns (every lane of the 16 gets it; ties keep the lower id).
// Every lane of the wave calls it.
template <bool COH>
__device__ __forceinline__ RowStat gemm_lm_panel(const GemmParams& a, int u, int ml, int n, bool rok, bool samp,
                                                 float rinv, float val, bool& nan_seen) {
  const int col = u * 16 + n;
  const bool valid = rok && col < a.V;
  const float lg = val * rinv;
  const Rsrc rl = make_rsrc(a.logits + (size_t)a.m0 * a.V, (uint32_t)((size_t)a.M * a.V * 4));
  st_f32<COH>(rl, valid ? (uint32_t)(ml * a.V + col) * 4u : kOob, lg);
  const bool isnan = lg != lg;
  nan_seen = nan_seen || (valid && isnan);
  const bool use = valid && !isnan;
  const float z = use ? (samp ? lg * a.inv_T : lg) : -INFINITY;
  const int id = use ? col : 0x7fffffff;
  float zm = z;
  int am = id;
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) {
    const float oz = __shfl_xor(zm, off);
    const int oa = __shfl_xor(am, off);
    const bool take = oz > zm || (oz == zm && oa < am);
    zm = take ? oz : zm;
    am = take ? oa : am;
  }
  float ex = (z == -INFINITY) ? 0.f : expf(z - zm);
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) ex += __shfl_xor(ex, off);
  return RowStat{zm, ex, am};
}

// Store a panel's statistics at pstats[m0 + ml][u] (lane n == 0 of the 16).
__device__ __forceinline__ void gemm_lm_store_panel(const GemmParams& a, int u, int ml, int n, bool rok,
                                                    const RowStat& ps) {
  const Rsrc rs = make_rsrc(a.pstats + (size_t)a.m0 * a.n_units * 3, (uint32_t)((size_t)a.M * a.n_units * 12));
  const uint32_t so = (rok && n == 0) ? (uint32_t)((ml * a.n_units + u) * 3) * 4u : kOob;
  st_f32<false>(rs, so, ps.m);
  st_f32<false>(rs, so == kOob ? kOob : so + 4u, ps.s);
  st_f32<false>(rs, so == kOob ? kOob : so + 8u, __int_as_float(ps.a));
}

// Sampling row?  (launch row ml of request (m0 + ml) / R)
__device__ __forceinline__ bool gemm_lm_samp(const GemmParams& a, int ml, bool rok) {
  if (!rok || a.mode == nullptr) return false;
  const int bl = (a.m0 + ml) / a.R;
  return a.mode[bl] == SPADE_SAMPLE && a.have_q;
}

// 1/rms of launch row `row` from the producer's per-16-column sums of
// squares: the sixteen threads sub = 0..15 of a row sum partials sub, sub + 16,
// ... in that order, then combine in a butterfly (all sixteen get the
// result).  Rows past M and launches without partials get 1.
__device__ __forceinline__ float gemm_row_rinv(const GemmParams& a, int row, int sub) {
  float s = 0.f;
  if (a.ssq_in != nullptr) {
    const Rsrc rs = make_rsrc(a.ssq_in + (size_t)a.m0 * a.n_ssq, (uint32_t)((size_t)a.M * a.n_ssq * 4));
    const uint32_t base = (uint32_t)(row * a.n_ssq) * 4u;
    const bool rok = row < a.M;
    for (int q0 = sub; q0 < a.n_ssq; q0 += 256) {
      float v[16];
#pragma unroll
      for (int f = 0; f < 16; ++f) {
        const int q = q0 + f * 16;
        v[f] = ld_f32<false>(rs, (rok && q < a.n_ssq) ? base + (uint32_t)q * 4u : kOob);
      }
#pragma unroll
      for (int f = 0; f < 16; ++f) s += v[f];
    }
  }
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  return (a.ssq_in != nullptr && row < a.M) ? 1.0f / sqrtf(s * a.inv_din + a.eps) : 1.0f;
}

// WBF16: bf16 weights (else f32); MT: 16-row tiles of activations (1 or 2);
// ALDS: activation operand copied to LDS once (MT == 1); COH: every output is
// a write-through (sc1) store and the residual stream is read with sc1 loads.
// Operands and row partials are read with plain loads: within one launch the
// caller gives every producer its own output region, so no L2 holds a stale
// line of them.
template <bool WBF16, int MT, bool ALDS, int KIND, bool COH>
struct Gemm {
  static constexpr int NW = kGemmWaves;
  static constexpr int S = WBF16 ? kActSplits : 1;
  static constexpr uint32_t ELT = WBF16 ? 2u : 4u;

  const GemmParams& a;
  GemmSmem<MT>& sm;
  uint8_t* lds_a;  // ALDS: operand copy (gemm_lds_a_bytes)
  int bid, G, tid, lane, wave;
  int NKB, nkw, kbl, cnt, T;
  // epilogue geometry of this thread: output row ml of the launch, column n of
  // the panel; tok: the thread holds a real output (tid < MT * 256)
  int ml, n, emtc, er;
  bool tok, rok;
  int pos, bg;  // QKV: position and request of row ml
  bool samp;    // LM: row ml uses 1/T statistics
  bool nan_seen;
  RowStat lmrun;  // LM: this workgroup's running (max, sum, argmax) of row ml over its units
  Rsrc ra[S];
  uint4 w0[8], w1[8], w2[8];
  uint4 av[MT][S][8];
  EpiIn e0, e1, e2;
  floatx4 acc[MT];

  __device__ __forceinline__ Gemm(const GemmParams& a_, GemmSmem<MT>& sm_, uint8_t* lds_a_, int bid_, int G_)
      : a(a_), sm(sm_), lds_a(lds_a_), bid(bid_), G(G_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    NKB = a.NKB;
    nkw = (NKB + NW - 1) / NW;
    kbl = (NKB * wave) / NW;
    cnt = (NKB * (wave + 1)) / NW - kbl;
    const int my_units = (a.n_units - bid + G - 1) / G;
    T = my_units * nkw;
    const int emt = tid >> 8;
    tok = emt < MT;
    emtc = tok ? emt : MT - 1;
    er = (tid >> 6) & 3;
    ml = emtc * 16 + 4 * (lane >> 4) + er;
    n = lane & 15;
    rok = tok && ml < a.M;
    nan_seen = false;
    lmrun = RowStat{-INFINITY, 0.f, 0x7fffffff};
    pos = 0;
    bg = 0;
    samp = false;
    if constexpr (KIND == GEMM_QKV || KIND == GEMM_LM) {
      const int m = a.m0 + ml;
      const int bl = m / a.R, i = m - bl * a.R;
      bg = a.b0 + bl;
      if constexpr (KIND == GEMM_QKV) {
        if (rok) pos = a.lens[bg] + i;
      } else {
        if (rok && a.mode != nullptr) samp = a.mode[bl] == SPADE_SAMPLE && a.have_q;
      }
    }
#pragma unroll
    for (int s = 0; s < S; ++s)
      ra[s] = make_rsrc((const uint8_t*)a.act + ((size_t)s * a.act_split + (size_t)a.m0 * a.act_stride) * ELT,
                        (uint32_t)((size_t)a.M * a.act_stride * ELT));
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // weight tile of item t (zeros past the stream or the wave's k-range)
  __device__ __forceinline__ void issue_w(int t, uint4 (&w)[8]) const {
    const int i = t / nkw, k = t - i * nkw;
    const bool ok = t < T && k < cnt;
    const int u = ok ? bid + i * G : 0;
    const uint8_t* tile = a.w + ((size_t)u * NKB + kbl + (ok ? k : 0)) * kTileBytes;
    const Rsrc r = make_rsrc(tile, ok ? (uint32_t)kTileBytes : 0u);
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = ld_stream_b128(r, (uint32_t)(lane * 16 + j * 1024));
  }

  // activation operand of k-block kbl + k (k >= cnt: zeros)
  __device__ __forceinline__ void issue_a_k(int k, uint4 (&dst)[MT][S][8]) const {
    const bool ok = k < cnt;
    const int kb = kbl + k;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int row = mt * 16 + (lane & 15);
      uint32_t off;
      if constexpr (WBF16) off = (uint32_t)(row * a.act_stride + kb * 256 + (lane >> 4) * 8) * 2u;
      else off = (uint32_t)(row * a.act_stride + kb * 128 + (lane >> 4) * 4) * 4u;
      off = ok ? off : kOob;
#pragma unroll
      for (int s = 0; s < S; ++s)
#pragma unroll
        for (int j = 0; j < 8; ++j) dst[mt][s][j] = ld_b128<false>(ra[s], off + (uint32_t)j * (WBF16 ? 64u : 64u));
    }
  }

  // activation operand of item t (streamed operand)
  __device__ __forceinline__ void issue_a_t(int t, uint4 (&dst)[MT][S][8]) const {
    const int i = t / nkw, k = t - i * nkw;
    issue_a_k(t < T ? k : cnt, dst);
  }

  // ALDS: copy rows [0, M) of every split into LDS with direct buffer->LDS
  // loads (no registers: each wave instruction moves 64 consecutive 16-byte
  // chunks of one row; rows are a multiple of 1 KB, gemm_lds_a_ok).  Nothing
  // else is written to LDS before the first wait, so the compiler's wait for
  // the copy (before any LDS access) leaves later loads in flight.
  __device__ __forceinline__ void fill_lds_a() {
    const uint32_t rowb = gemm_lds_row_bytes(a.act_stride, WBF16);
    const int row_bytes = a.act_stride * (int)ELT;
    const int per_row = row_bytes >> 10;  // wave instructions per row
    const int per_split = a.M * per_row;
    for (int i = wave; i < S * per_split; i += NW) {
      const int s = i / per_split, rem = i - s * per_split;
      const int row = rem / per_row, blk = rem - row * per_row;
      const Rsrc rs = (S == 1 || s == 0) ? ra[0] : ra[S - 1];  // no dynamic index into ra
      __attribute__((address_space(3))) void* dst =
          (__attribute__((address_space(3))) void*)(lds_a + (uint32_t)(s * a.M + row) * rowb + (uint32_t)blk * 1024u);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 16, (uint32_t)(row * row_bytes + blk * 1024 + lane * 16), 0, 0, 0);
    }
  }

  // ALDS: fragment of k-block kbl + k for this lane (k >= cnt reads block kbl:
  // finite values that meet a zero weight tile)
  __device__ __forceinline__ void read_a_lds(int k) {
    const uint32_t rowb = gemm_lds_row_bytes(a.act_stride, WBF16);
    const int r = lane & 15;
    const int rr = r < a.M ? r : a.M - 1;
    const int kb = kbl + (k < cnt ? k : 0);
    uint32_t off;
    if constexpr (WBF16) off = (uint32_t)rr * rowb + (uint32_t)(kb * 256 + (lane >> 4) * 8) * 2u;
    else off = (uint32_t)rr * rowb + (uint32_t)(kb * 128 + (lane >> 4) * 4) * 4u;
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        av[0][s][j] = *(const uint4*)(lds_a + (uint32_t)(s * a.M) * rowb + off + (uint32_t)j * 64u);
  }

  // epilogue inputs of the unit of item t
  __device__ __forceinline__ EpiIn epi_load(int t) const {
    return gemm_epi_load<KIND, COH>(a, bid + (t / nkw) * G, ml, n, rok && t < T, pos);
  }

  __device__ __forceinline__ void mma(const uint4 (&w)[8], const uint4 (&x)[MT][S][8]) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if constexpr (WBF16) {
#pragma unroll
          for (int s = S - 1; s >= 0; --s)
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x[mt][s][j]),
                                                              __builtin_bit_cast(bf16x8, w[j]), acc[mt], 0, 0, 0);
        } else {
          const float4 w4 = __builtin_bit_cast(float4, w[j]);
          const float4 a4 = __builtin_bit_cast(float4, x[mt][0][j]);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.x, w4.x, acc[mt], 0, 0, 0);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.y, w4.y, acc[mt], 0, 0, 0);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.z, w4.z, acc[mt], 0, 0, 0);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.w, w4.w, acc[mt], 0, 0, 0);
        }
      }
  }

  // Epilogue of unit u for this thread's output (row ml, column n): val is
  // the full dot product.  D[i][j] of a 16x16 MFMA sits in lane j + 16*(i/4),
  // register i%4.
  __device__ __forceinline__ void epilogue(int u, float val, const EpiIn& e) {
    const float rinv = sm.rinv[ml];
    if constexpr (KIND != GEMM_LM) {
      gemm_epilogue<KIND, WBF16, COH>(a, u, ml, n, rok, pos, bg, rinv, val, e);
    } else {  // GEMM_LM: logits and the panel's (max, sum exp, argmax) of z = logit / T
      // fold the panel into this workgroup's running statistics of the row
      // (panels in the workgroup's unit order); stored once after the loop
      const RowStat ps = gemm_lm_panel<COH>(a, u, ml, n, rok, samp, rinv, val, nan_seen);
      if (ps.m != -INFINITY) lmrun = merge_stat(lmrun, ps);
    }
  }

  __device__ __forceinline__ void unit_end(int t, const EpiIn& e) {
    const int u = bid + (t / nkw) * G;
    const bool keep = rok;
    rok = rok && t < T;  // padding units store nothing
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) sm.red[wave][mt][r][lane] = acc[mt][r];
    __syncthreads();
    float val = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) val += sm.red[w][emtc][er][lane];
    epilogue(u, val, e);
    rok = keep;
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // 1/rms of every row from the producer's per-16-column sums of squares:
  // thread (row, sub) sums partials sub, sub + 16, ... in that order, then the
  // sixteen subs combine in a butterfly.  The first 32 partials of each thread
  // (d <= 8192; 16 with two row tiles, for registers) are requested with the
  // other prologue loads (ssq_issue).
  static constexpr int kSsqFirst = MT == 1 ? 32 : 16;

  __device__ __forceinline__ Rsrc ssq_rsrc() const {
    return make_rsrc(a.ssq_in + (size_t)a.m0 * a.n_ssq, (uint32_t)((size_t)a.M * a.n_ssq * 4));
  }

  __device__ __forceinline__ void ssq_issue(float (&v)[kSsqFirst]) const {
    const int row = tid >> 4, sub = tid & 15;
    const Rsrc rs = ssq_rsrc();
    const uint32_t base = (uint32_t)(row * a.n_ssq) * 4u;
#pragma unroll
    for (int f = 0; f < kSsqFirst; ++f) {
      const int q = sub + f * 16;
      v[f] = ld_f32<false>(rs, (a.ssq_in != nullptr && q < a.n_ssq) ? base + (uint32_t)q * 4u : kOob);
    }
  }

  __device__ __forceinline__ void row_scales(const float (&v0)[kSsqFirst]) {
    const int row = tid >> 4, sub = tid & 15;
    float s = 0.f;
#pragma unroll
    for (int f = 0; f < kSsqFirst; ++f) s += v0[f];
    if (a.ssq_in != nullptr) {
      const Rsrc rs = ssq_rsrc();
      const uint32_t base = (uint32_t)(row * a.n_ssq) * 4u;
      for (int q0 = sub + 16 * kSsqFirst; q0 < a.n_ssq; q0 += 256) {
        float v[16];
#pragma unroll
        for (int f = 0; f < 16; ++f) {
          const int q = q0 + f * 16;
          v[f] = ld_f32<false>(rs, q < a.n_ssq ? base + (uint32_t)q * 4u : kOob);
        }
#pragma unroll
        for (int f = 0; f < 16; ++f) s += v[f];
      }
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) s += __shfl_xor(s, off);
    if (sub == 0 && row < MT * 16)
      sm.rinv[row] = (a.ssq_in != nullptr && row < a.M) ? 1.0f / sqrtf(s * a.inv_din + a.eps) : 1.0f;
  }

  template <int P>
  __device__ __forceinline__ void step(int t) {
    if constexpr (P == 0) step_impl(t, w0, e0, e2);
    else if constexpr (P == 1) step_impl(t, w1, e1, e0);
    else step_impl(t, w2, e2, e1);
  }

  // item t: consume tile w, refill it with item t + 3, fetch the epilogue
  // inputs of item t + 2 into enew, finish the unit with ecur
  __device__ __forceinline__ void step_impl(int t, uint4 (&w)[8], EpiIn& ecur, EpiIn& enew) {
    const int k = t - (t / nkw) * nkw;
    // a padding item (t >= T, the same in every wave) only keeps the loads'
    // count: its MFMAs and its unit's sum would be discarded
    const bool live = t < T;
    if (live) {
      if constexpr (ALDS) read_a_lds(k);
      mma(w, av);
    }
    // the refills below reuse the registers just consumed: keep them after
    // the MFMAs so no fourth tile is ever live
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!ALDS) issue_a_t(t + 1, av);
    issue_w(t + 3, w);
    enew = epi_load(t + 2);
    if (live && k == nkw - 1) unit_end(t, ecur);
  }

  // The item loop (no exits inside; the item count is padded to a multiple of
  // 3 with padding items that load zeros and store nothing, so the wait
  // counts at the loop head stay exact).
  __device__ __forceinline__ void items() {
    const int Tpad = (T + 2) / 3 * 3;
    for (int t = 0; t < Tpad; t += 3) {
      step<0>(t);
      step<1>(t + 1);
      step<2>(t + 2);
    }
  }

  // The whole launch: operands, row scales, the item loop.  Request order
  // (scheduling barriers keep it): weight tiles 0 and 1, the operand copy, the
  // epilogue inputs and the row partials, weight tile 2.  Every workgroup
  // starts at once, so whatever is requested behind the first weight tiles
  // queues behind the whole chip's: the operand comes after two tiles (it
  // waited behind three before, or the weights behind the operand: both
  // measured slower).  Loads complete in issue order, so the prologue waits
  // for all but tile 2's eight loads, and the loop starts with a tile in
  // flight.
  __device__ __forceinline__ void run() {
    issue_w(0, w0);
    issue_w(1, w1);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (ALDS) fill_lds_a();
    else issue_a_t(0, av);
    e0 = epi_load(0);
    e1 = epi_load(1);
    float sv[kSsqFirst];
    ssq_issue(sv);
    __builtin_amdgcn_sched_barrier(0);
    issue_w(2, w2);
    __builtin_amdgcn_sched_barrier(0);
    row_scales(sv);
    wait_vmcnt<8>();
    __syncthreads();
    items();
    finish();
  }

  __device__ __forceinline__ void finish() {
    if constexpr (KIND == GEMM_LM) {
      // one (max, sum exp, argmax) per (row, workgroup): stats[m][bid], NU = grid size
      const Rsrc rst = make_rsrc(a.stats + (size_t)a.m0 * a.NU * 3, (uint32_t)((size_t)a.M * a.NU * 12));
      const uint32_t so = (rok && n == 0) ? (uint32_t)((ml * a.NU + bid) * 3) * 4u : kOob;
      st_f32<COH>(rst, so, lmrun.m);
      st_f32<COH>(rst, so == kOob ? kOob : so + 4u, lmrun.s);
      st_f32<COH>(rst, so == kOob ? kOob : so + 8u, __int_as_float(lmrun.a));
    }
    if (nan_seen) flag_error(a.err, SPADE_DERR_NAN);
  }
};

}  // namespace spade
