// Split-K skinny GEMM for the projections (QKV, O, gate/up, down) and the LM
// head when the activation operand (<= 16 rows) is too long for one LDS copy:
// the down projection at 7B (6 rows x 11008 x two bf16 terms = 264 KB) and
// every projection at 13B.  The LM head stores per-panel statistics, as in
// the wide-row engine.  The skinny engine (device_gemm.h) then has to fetch the
// operand from L2 with every weight tile, one tile ahead, and waits on that
// round trip at every step.
//
// Here the K range is cut into KS k-splits along the engine's eight k-ranges
// (split s: ranges [8s/KS, 8(s+1)/KS)).  Workgroup b belongs to k-split
// b / G (G = grid / KS) and copies only that split's k-blocks of the operand
// into LDS, once, with direct buffer->LDS loads.  It then walks panel groups
// j, j + G, ... (j = b % G) of KS panels each: wave w takes panel w / (8/KS) of
// the group and k-range w % (8/KS) of its split, so each wave streams one
// k-range of one panel per group through the same three-deep register
// pipeline as the skinny engine, reading the operand from LDS.
//
// Sums: the arithmetic contract of every engine is total = 0 + r0 + r1 + ...
// + r7 in range order, each range r a fresh MFMA accumulator over its
// k-blocks in order.  At the end of a group the workgroup of split 0 adds its
// ranges in that order and publishes the running sum; the other splits
// publish their range partials one by one (write-through stores).  After the
// item loop each workgroup arrives on the counter of each of its groups; the
// last arrival continues the sum over the remaining ranges in order and runs
// the kind's epilogue.  Results are bit-identical to the skinny and wide-row
// engines.
#pragma once

#include "device_gemm.h"

namespace spade {

constexpr int kSplitMaxGroups = 64;  // panel groups per workgroup (host-checked)

struct GemmSplitSmem {
  float red[kGemmWaves][4][64];
  float rinv[16];
  int last[kSplitMaxGroups];
};

// LDS row of the operand copy of one k-split: whole 1 KB blocks (two
// k-blocks) plus 16 bytes, so rows start 4 banks apart.
inline __host__ __device__ uint32_t gemm_split_row_bytes(int nkbs) { return (uint32_t)((nkbs + 1) / 2) * 1024u + 16u; }
inline __host__ __device__ int gemm_split_max_kblocks(int NKB, int KS) {
  int mx = 0;
  for (int s = 0; s < KS; ++s) {
    const int n = (NKB * (s + 1)) / KS - (NKB * s) / KS;
    mx = n > mx ? n : mx;
  }
  return mx;
}
inline __host__ __device__ uint32_t gemm_split_lds_bytes(int M, int NKB, int KS) {
  return (uint32_t)kActSplits * (uint32_t)M * gemm_split_row_bytes(gemm_split_max_kblocks(NKB, KS));
}

// KS: k-splits (2 or 4); bf16 weights, one 16-row tile of activations.
template <int KS, int KIND>
struct GemmSplit {
  static constexpr int NW = kGemmWaves;
  static constexpr int S = kActSplits;
  static constexpr int RPS = NW / KS;  // k-ranges per split = waves per panel
  static_assert(KS == 2 || KS == 4, "k-splits");

  const GemmParams& a;
  GemmSplitSmem& sm;
  uint8_t* lds_a;
  uint32_t* cnt;  // [groups] arrival counters (zero between launches)
  float* part;    // [n_units][8][256] published sums and range partials
  int tid, lane, wave, G, ks, j;
  int NKB, nkw, kbl, cnt_k, kb0, nkbs, T, ui, n_groups, my_groups;
  uint32_t rowb;
  Rsrc ra[S];
  uint4 w0[8], w1[8], w2[8];
  uint4 av[S][8];
  floatx4 acc;

  __device__ __forceinline__ GemmSplit(const GemmParams& a_, GemmSplitSmem& sm_, uint8_t* lds_a_, uint32_t* cnt_,
                                       float* part_, int G_)
      : a(a_), sm(sm_), lds_a(lds_a_), cnt(cnt_), part(part_), G(G_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int b = (int)blockIdx.x;
    ks = b / G;
    j = b - ks * G;
    NKB = a.NKB;
    nkw = (NKB + NW - 1) / NW;
    ui = wave / RPS;
    const int r = ks * RPS + wave % RPS;  // this wave's k-range
    kbl = (NKB * r) / NW;
    cnt_k = (NKB * (r + 1)) / NW - kbl;
    kb0 = (NKB * ks) / KS;
    nkbs = (NKB * (ks + 1)) / KS - kb0;
    rowb = gemm_split_row_bytes(nkbs);
    n_groups = (a.n_units + KS - 1) / KS;
    my_groups = j < n_groups ? (n_groups - j + G - 1) / G : 0;
    T = my_groups * nkw;
#pragma unroll
    for (int s = 0; s < S; ++s)
      ra[s] = make_rsrc((const uint8_t*)a.act + ((size_t)s * a.act_split + (size_t)a.m0 * a.act_stride) * 2,
                        (uint32_t)((size_t)a.M * a.act_stride * 2));
    acc = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // weight tile of item t: group i = t / nkw, k-block kbl + t % nkw of this
  // wave's panel (zeros past the stream, the range or the last panel)
  __device__ __forceinline__ void issue_w(int t, uint4 (&w)[8]) const {
    const int i = t / nkw, k = t - i * nkw;
    const int u = (j + i * G) * KS + ui;
    const bool ok = t < T && k < cnt_k && u < a.n_units;
    const uint8_t* tile = a.w + ((size_t)(ok ? u : 0) * NKB + kbl + (ok ? k : 0)) * kTileBytes;
    const Rsrc r = make_rsrc(tile, ok ? (uint32_t)kTileBytes : 0u);
#pragma unroll
    for (int q = 0; q < 8; ++q) w[q] = ld_stream_b128(r, (uint32_t)(lane * 16 + q * 1024));
  }

  // copy k-blocks [kb0, kb0 + nkbs) of rows 0..M-1 of every split into LDS:
  // one wave instruction moves 1 KB (two k-blocks) of one row; an odd count
  // moves one k-block past the split, into the row's padding block (rows end
  // past the buffer read zeros)
  __device__ __forceinline__ void fill_lds_a() {
    const int per_row = (nkbs + 1) / 2;
    const int per_split = a.M * per_row;
    for (int i = wave; i < S * per_split; i += NW) {
      const int s = i / per_split, rem = i - s * per_split;
      const int row = rem / per_row, blk = rem - row * per_row;
      const Rsrc rs = s == 0 ? ra[0] : ra[S - 1];
      __attribute__((address_space(3))) void* dst =
          (__attribute__((address_space(3))) void*)(lds_a + (uint32_t)(s * a.M + row) * rowb + (uint32_t)blk * 1024u);
      const uint32_t off = (uint32_t)(row * a.act_stride + kb0 * 256) * 2u + (uint32_t)blk * 1024u + (uint32_t)lane * 16u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 16, off, 0, 0, 0);
    }
  }

  // operand fragment of k-block kbl + k (k >= cnt_k reads kbl: finite values
  // that meet a zero weight tile); rows past M read row M - 1, whose products
  // are never stored
  __device__ __forceinline__ void read_a_lds(int k) {
    const int r = lane & 15;
    const int rr = r < a.M ? r : a.M - 1;
    const int kb = kbl + (k < cnt_k ? k : 0) - kb0;
    const uint32_t off = (uint32_t)rr * rowb + (uint32_t)(kb * 256 + (lane >> 4) * 8) * 2u;
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int q = 0; q < 8; ++q)
        av[s][q] = *(const uint4*)(lds_a + (uint32_t)(s * a.M) * rowb + off + (uint32_t)q * 64u);
  }

  __device__ __forceinline__ void mma(const uint4 (&w)[8]) {
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int s = S - 1; s >= 0; --s)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av[s][q]),
                                                      __builtin_bit_cast(bf16x8, w[q]), acc, 0, 0, 0);
  }

  // Output o (0 .. KS*256-1) of a group: panel o / 256 of the group, MFMA
  // register (o / 64) % 4, lane o % 64 -> row 4 (lane / 16) + register,
  // column lane % 16.  Thread tid handles o = tid + 512 q.
  static constexpr int OPT = KS * 256 / 512;  // outputs per thread

  // end of group i: sums of this split's ranges in range order; split 0
  // publishes its running sum in slot 0, the others each range r in slot r
  __device__ __forceinline__ void group_end(int t) {
    const int i = t / nkw;
    const int grp = j + i * G;
    const bool real = t < T;
#pragma unroll
    for (int r = 0; r < 4; ++r) sm.red[wave][r][lane] = acc[r];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < OPT; ++q) {
      const int o = tid + 512 * q;
      const int pu = o >> 8, er = (o >> 6) & 3;
      const int ml = 4 * (lane >> 4) + er, n = lane & 15;
      const int u = grp * KS + pu;
      const bool ok = real && ml < a.M && u < a.n_units;
      float* pp = part + ((size_t)u * 8) * 256 + ml * 16 + n;
      if (ks == 0) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < RPS; ++w) s += sm.red[pu * RPS + w][er][lane];
        if (ok) __hip_atomic_store(pp, s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {
#pragma unroll
        for (int w = 0; w < RPS; ++w) {
          const int r = ks * RPS + w;
          if (ok) __hip_atomic_store(pp + r * 256, sm.red[pu * RPS + w][er][lane], __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
    __syncthreads();
    acc = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  template <int P>
  __device__ __forceinline__ void step(int t) {
    if constexpr (P == 0) step_impl(t, w0);
    else if constexpr (P == 1) step_impl(t, w1);
    else step_impl(t, w2);
  }

  __device__ __forceinline__ void step_impl(int t, uint4 (&w)[8]) {
    const int k = t - (t / nkw) * nkw;
    // a padding item (t >= T, the same in every wave) only keeps the loads'
    // count: its MFMAs and its group's sum would be discarded
    const bool live = t < T;
    if (live) {
      read_a_lds(k);
      mma(w);
    }
    __builtin_amdgcn_sched_barrier(0);
    issue_w(t + 3, w);
    if (live && k == nkw - 1) group_end(t);
  }

  // the last arrival of group grp: continue split 0's running sum over the
  // ranges of the other splits in order, then the epilogue
  __device__ __forceinline__ void finish(int grp) {
    const Rsrc rp = make_rsrc(part, 0x7ffffff0u);
#pragma unroll
    for (int q = 0; q < OPT; ++q) {
      const int o = tid + 512 * q;
      const int pu = o >> 8, er = (o >> 6) & 3;
      const int ml = 4 * (lane >> 4) + er, n = lane & 15;
      const int u = grp * KS + pu;
      const bool uok = u < a.n_units;
      const bool rok = uok && ml < a.M;
      const uint32_t base = (uint32_t)(((size_t)(uok ? u : 0) * 8) * 256 + ml * 16 + n) * 4u;
      float v[8];
#pragma unroll
      for (int r = 0; r < 8; ++r)
        v[r] = (r == 0 || r >= RPS) ? ld_b32_coh(rp, rok ? base + (uint32_t)r * 1024u : kOob) : 0.f;
      float val = v[0];
#pragma unroll
      for (int r = RPS; r < 8; ++r) val += v[r];
      if constexpr (KIND == GEMM_LM) {
        const bool samp = gemm_lm_samp(a, ml, rok);
        bool nan_seen = false;
        const RowStat ps = gemm_lm_panel<false>(a, uok ? u : 0, ml, n, rok, samp, sm.rinv[ml], val, nan_seen);
        gemm_lm_store_panel(a, uok ? u : 0, ml, n, rok, ps);
        if (nan_seen) flag_error(a.err, SPADE_DERR_NAN);
      } else {
        int pos = 0, bg = 0;
        if constexpr (KIND == GEMM_QKV) {
          const int m = a.m0 + ml;
          const int bl = m / a.R, ir = m - bl * a.R;
          bg = a.b0 + bl;
          if (rok) pos = a.lens[bg] + ir;
        }
        const EpiIn e = gemm_epi_load<KIND, false>(a, uok ? u : 0, ml, n, rok, pos);
        gemm_epilogue<KIND, true, false>(a, uok ? u : 0, ml, n, rok, pos, bg, sm.rinv[ml], val, e);
      }
    }
  }

  // Request order: weight tile 0, this split's operand copy, weight tiles 1
  // and 2 (the operand waits behind one tile of every workgroup's instead of
  // three); the prologue waits for all but tiles 1 and 2.
  __device__ __forceinline__ void run() {
    issue_w(0, w0);
    __builtin_amdgcn_sched_barrier(0);
    fill_lds_a();
    __builtin_amdgcn_sched_barrier(0);
    issue_w(1, w1);
    issue_w(2, w2);
    __builtin_amdgcn_sched_barrier(0);
    for (int r = tid >> 4; r < 16; r += 32) {
      const float ri = gemm_row_rinv(a, r, tid & 15);
      if ((tid & 15) == 0) sm.rinv[r] = ri;
    }
    wait_vmcnt<16>();
    __syncthreads();
    // item count padded to a multiple of 3 with no exits inside the loop
    const int Tpad = (T + 2) / 3 * 3;
    for (int t = 0; t < Tpad; t += 3) {
      step<0>(t);
      step<1>(t + 1);
      step<2>(t + 2);
    }
    // every published value has landed: arrive on each group's counter
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid < my_groups) {
      const int grp = j + tid * G;
      const uint32_t old = __hip_atomic_fetch_add(cnt + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int last = old == (uint32_t)KS - 1u;
      if (last) __hip_atomic_store(cnt + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      sm.last[tid] = last;
    }
    __syncthreads();
    for (int i = 0; i < my_groups; ++i)
      if (sm.last[i]) finish(j + i * G);  // uniform across the workgroup
  }
};

}  // namespace spade
