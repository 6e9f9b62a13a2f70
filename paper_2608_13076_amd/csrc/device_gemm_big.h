// Compute-bound GEMM for the projections of prefill forwards (hundreds to
// thousands of rows; Sec. III-A: every prompt token goes through the whole
// verifier once): QKV, O, gate/up and down with the wide-row engine's
// epilogues.
//
// A workgroup of 8 waves (two per SIMD) owns 128 rows (8 row tiles) and 16
// panels (256 columns); wave w takes row tiles 4 (w % 2) .. + 3 and panels
// 4 (w / 2) .. + 3: 16 MFMA output tiles, each with a running k-range
// accumulator and a total.  The k-loop runs in 32-k slices (one MFMA k-step;
// 8 per 256-k block).  A slice of the activations (128 rows x 32 k x two
// bf16 terms, 16 KB) goes by direct buffer->LDS loads into a five-slot ring,
// four slices ahead; each wave reads its row tiles' fragments (inline-asm
// ds_read_b128 with explicit waits, so the compiler does not wait for the
// fills in flight), each feeding 4 MFMAs.  The weight fragments of a slice
// (1 KB per panel, 16 bytes per lane, contiguous in the arena's tiles) load
// straight into a four-slice register ring.  Each weight byte is multiplied
// with 128 rows per workgroup and each activation byte in LDS with 64
// columns per read: per 32 MFMAs a wave moves 6 KB from L2 and reads 8 KB of
// LDS.
//
// Arithmetic is the skinny engine's, operation for operation: per output,
// the k-blocks of each of the eight k-ranges (range r: k-blocks
// [NKB r / 8, NKB (r + 1) / 8)) accumulate in a fresh MFMA accumulator, slice
// by slice, the low bf16 term of the activation before the high one; the
// range partials are added to the total in range order.  A row's result does
// not depend on the engine or on the other rows.
#pragma once

#include "device_gemm.h"

namespace spade {

constexpr int kBigWaves = 8;
constexpr int kBigRows = 128;   // rows per workgroup (8 row tiles)
constexpr int kBigRT = kBigRows / 16;           // row tiles per workgroup
constexpr int kBigRowWaves = kBigRT / 4;        // waves across the rows (4 row tiles each)
static_assert(kBigWaves == 4 * kBigRowWaves, "4 panel groups of waves");
constexpr int kBigUnits = 16;   // panels per workgroup (4 per wave)
constexpr int kBigSlots = 5;    // activation slices in the LDS ring
constexpr int kBigDepth = 4;    // slices requested ahead of the one in use

struct GemmBigSmem {
  union {
    // slot, split, row tile: 16 rows x 64 bytes, the four 16-byte pieces of
    // row r at piece p ^ f(r), f(r) = ((r / 2) ^ (r / 4)) % 4: the rows of a
    // fragment read that share a pass (8 consecutive rows with 32 banks, or
    // rows r, r + 4, r + 8, r + 12 with 64) land on distinct banks
    uint8_t ring[kBigSlots][kActSplits][kBigRT][1024];
    // after the k-loop: each lane's totals, [wave][row tile][panel][lane]
    floatx4 tot[kBigWaves][4][4][64];
  };
  float rinv[kBigRows];
};

typedef uint32_t u32x4b __attribute__((ext_vector_type(4)));

template <int KIND>
struct GemmBig {
  static_assert(KIND != GEMM_LM, "projections only");
  static constexpr int S = kActSplits;
  static constexpr int D = kBigDepth;
  const GemmParams& a;
  GemmBigSmem& sm;
  int tid, lane, wave, g, kl;
  int row0, u0;        // first row of the workgroup, first panel of this wave
  int mt0;             // first row tile of this wave
  int NKB;
  uint32_t lds_ring;   // LDS byte address of the ring
  uint32_t frag_off;   // this lane's fragment offset within a 1 KB block
  Rsrc ract;           // activations of this launch's rows, both splits
  Rsrc rw[4];          // this wave's weight panels (empty past n_units)
  floatx4 acc[4][4], tot[4][4];
  uint4 wq[D][4];      // weight fragments of the slices in flight
  int rnext, bnd;      // next k-range, its first k-block
  int T;               // slices of the k-loop

  __device__ __forceinline__ GemmBig(const GemmParams& a_, GemmBigSmem& sm_, int rg, int ug) : a(a_), sm(sm_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    g = lane >> 4;
    kl = lane & 15;
    row0 = rg * kBigRows;
    mt0 = 4 * (wave % kBigRowWaves);
    u0 = ug * kBigUnits + (wave / kBigRowWaves) * 4;
    NKB = a.NKB;
    T = NKB * 8;
    lds_ring = (uint32_t)(size_t)(__attribute__((address_space(3))) void*)&sm.ring[0][0][0][0];
    frag_off = (uint32_t)(kl * 64 + 16 * (g ^ (((kl >> 1) ^ (kl >> 2)) & 3)));
    ract = make_rsrc((const uint8_t*)a.act + (size_t)a.m0 * a.act_stride * 2,
                     (uint32_t)(((size_t)(S - 1) * a.act_split + (size_t)a.M * a.act_stride) * 2));
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int u = u0 + p;
      const bool ok = u < a.n_units;
      rw[p] = make_rsrc(a.w + (size_t)(ok ? u : 0) * NKB * kTileBytes, ok ? (uint32_t)(NKB * kTileBytes) : 0u);
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        acc[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
        tot[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
    rnext = 1;
    bnd = NKB / kGemmWaves;
    while (bnd == 0 && rnext < kGemmWaves) bnd = (NKB * ++rnext) / kGemmWaves;
  }

  // Request slice t (k-block t / 8, k-step t % 8) of the activations into
  // ring slot t % kBigSlots: each wave moves two of the 16 (split, row tile)
  // blocks, one 16-byte piece per lane (lane l: row l / 4, piece l % 4 of the
  // swizzled block).  Rows past M repeat row M - 1: finite values whose
  // products are never stored.  Slices past the k-loop read zeros (an offset
  // past the resource) into a slot no later slice reads: every load is
  // issued unconditionally, so the compiler's wait counts stay exact.
  __device__ __forceinline__ void fill(int t) const {
    const int kb = t >> 3, j = t & 7;
    const int slot = t % kBigSlots;
    const int r = lane >> 2, pp = lane & 3;
    const int lp = pp ^ (((r >> 1) ^ (r >> 2)) & 3);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = wave * 2 + i;
      const int s = q / kBigRT, mt = q % kBigRT;
      const int row = row0 + mt * 16 + r;
      const int grow = row < a.M ? row : a.M - 1;
      const uint32_t off =
          t < T ? (uint32_t)(((size_t)s * a.act_split + (size_t)grow * a.act_stride + kb * 256 + j * 32 + lp * 8) * 2)
                : kOob;
      __attribute__((address_space(3))) void* dst =
          (__attribute__((address_space(3))) void*)&sm.ring[slot][s][mt][0];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ract, dst, 16, off, 0, 0, 0);
    }
  }

  // weight fragments of slice t for this wave's four panels (zeros past the
  // k-loop: the offset is past the resource)
  __device__ __forceinline__ void issue_w(int t, uint4 (&w)[4]) const {
    const uint32_t off = t < T ? (uint32_t)((t >> 3) * kTileBytes + (t & 7) * 1024 + lane * 16) : kOob;
#pragma unroll
    for (int p = 0; p < 4; ++p) w[p] = ld_b128<false>(rw[p], off);
  }

  template <int OFF>
  __device__ __forceinline__ static u32x4b ds_read16(uint32_t addr) {
    u32x4b v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
  }

  template <int... MT>
  __device__ __forceinline__ static void read_frags(uint32_t base, u32x4b (&x)[4][S], std::integer_sequence<int, MT...>) {
    ((x[MT][0] = ds_read16<MT * 1024>(base), x[MT][1] = ds_read16<kBigRT * 1024 + MT * 1024>(base)), ...);
  }

  // wait until at most N of this wave's LDS reads are outstanding; the
  // fragments x depend on the wait
  template <int N>
  __device__ __forceinline__ static void lds_wait_n(u32x4b (&x)[S]) {
#pragma unroll
    for (int s = 0; s < S; ++s) asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x[s]) : "n"(N));
  }

  // the MFMAs of slice t: fragments of its ring slot (this wave's row
  // tiles), weights w
  __device__ __forceinline__ void mma(int t, const uint4 (&w)[4]) {
    const uint32_t base =
        lds_ring + (uint32_t)(t % kBigSlots) * (uint32_t)(S * kBigRT * 1024) + (uint32_t)mt0 * 1024u + frag_off;
    u32x4b x[4][S];
    read_frags(base, x, std::make_integer_sequence<int, 4>{});
    // row tile mt's two fragments are the reads 2 mt and 2 mt + 1 of eight:
    // its MFMAs start once those have landed (LDS reads complete in order)
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt == 0) lds_wait_n<6>(x[0]);
      else if (mt == 1) lds_wait_n<4>(x[1]);
      else if (mt == 2) lds_wait_n<2>(x[2]);
      else lds_wait_n<0>(x[3]);
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int s = S - 1; s >= 0; --s)
          acc[mt][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x[mt][s]),
                                                               __builtin_bit_cast(bf16x8, w[p]), acc[mt][p], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);  // keep row tile mt's MFMAs before the next wait
    }
  }

  // after k-block kb: at the end of a k-range add its partial to the total
  __device__ __forceinline__ void range_end(int kb) {
    if (kb + 1 == bnd) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int p = 0; p < 4; ++p) {
#pragma unroll
          for (int i = 0; i < 4; ++i) tot[mt][p][i] += acc[mt][p][i];
          acc[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
      do {
        ++rnext;
        bnd = (NKB * rnext) / kGemmWaves;
      } while (bnd == kb + 1 && rnext < kGemmWaves);
    }
  }

  // slice t = 8 kb + J: wait for this wave's share of its fill and for its
  // weights (the D - 1 slices after it have their six loads each in flight),
  // publish the slot to every wave (bare barrier: the ring is read with
  // inline asm and written by direct loads each wave has waited for),
  // request slice t + D into slot (t + D) % kBigSlots -- the slot of slice
  // t - 1, which every wave finished reading before this barrier -- then the
  // MFMAs, then the weights of slice t + D into the registers just used.
  template <int J>
  __device__ __forceinline__ void slice(int kb) {
    const int t = kb * 8 + J;
    wait_vmcnt<(D - 1) * 6>();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    fill(t + D);
    mma(t, wq[J % D]);
    __builtin_amdgcn_sched_barrier(0);
    issue_w(t + D, wq[J % D]);
  }

  template <int... I>
  __device__ __forceinline__ void kblock(int kb, std::integer_sequence<int, I...>) {
    (slice<I>(kb), ...);
  }

  __device__ __forceinline__ void run() {
    // prologue: the first D slices (each one fill, then its weights: the
    // waits count two fill loads and four weight loads per slice)
#pragma unroll
    for (int i = 0; i < D; ++i) {
      fill(i);
      issue_w(i, wq[i]);
    }
    for (int kb = 0; kb < NKB; ++kb) {
      kblock(kb, std::make_integer_sequence<int, 8>{});
      range_end(kb);
    }
    // the ring is idle once every fill has landed and every wave is past its
    // last read: the totals move to LDS, so the epilogue runs as a loop
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int p = 0; p < 4; ++p) sm.tot[wave][mt][p][lane] = tot[mt][p];
    for (int r = tid >> 4; r < kBigRows; r += kBigWaves * 4) {
      const float ri = gemm_row_rinv(a, row0 + r, tid & 15);
      if ((tid & 15) == 0) sm.rinv[r] = ri;
    }
    __syncthreads();
    // epilogue: lane holds rows mt*16 + 4g + i, column kl of each panel
#pragma unroll 1
    for (int q = 0; q < 16; ++q) {
      const int mt = q >> 2, p = q & 3;
      const int u = u0 + p;
      const bool uok = u < a.n_units;
      const floatx4 v = sm.tot[wave][mt][p][lane];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = (mt0 + mt) * 16 + 4 * g + i;
        const int ml = row0 + r;
        const bool rok = uok && ml < a.M;
        int pos = 0, bg = 0;
        if constexpr (KIND == GEMM_QKV) {
          const int m = a.m0 + ml;
          const int bl = m / a.R, ir = m - bl * a.R;
          bg = a.b0 + bl;
          if (rok) pos = a.lens[bg] + ir;
        }
        const EpiIn e = gemm_epi_load<KIND, false>(a, uok ? u : 0, ml, kl, rok, pos);
        gemm_epilogue<KIND, true, false>(a, uok ? u : 0, ml, kl, rok, pos, bg, sm.rinv[r], v[i], e);
      }
    }
  }
};

// Host-side shape of a launch: row groups, panel groups; workgroups
// 8 * ceil(panel groups / 8) * row groups (the row groups of one panel group
// share an XCD and its L2).
inline __host__ __device__ int gemm_big_row_groups(int M) { return (M + kBigRows - 1) / kBigRows; }
inline __host__ __device__ int gemm_big_unit_groups(int n_units) { return (n_units + kBigUnits - 1) / kBigUnits; }

}  // namespace spade
