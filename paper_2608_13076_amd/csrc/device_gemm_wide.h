// Wide-row GEMM for the projection kinds (QKV, O, gate/up, down) when the
// activation operand has more rows than the skinny engine (device_gemm.h)
// keeps resident: batched verification, M = B (gamma + 1) up to 256 rows.
//
// A workgroup of 8 waves owns 8 consecutive panels ("units"), one per wave,
// and a group of RT 16-row tiles.  Each wave streams its panel's k-blocks
// (8 KB weight tiles) through the same three-deep register pipeline as the
// skinny engine and multiplies every tile with all RT row tiles.  The
// activation k-block (RT * 16 rows x 256 k, two bf16 terms) is shared by the
// eight waves through a two-slot LDS ring: each thread loads its share of
// k-block kb + 3 into registers (two staging sets), writes k-block kb + 1
// into the free slot after the MFMAs of kb, and one barrier per k-block
// publishes it.  The loads of a step are issued activation first, weights
// second, so the wait for the activation block never waits for a weight tile
// issued after it.
//
// Row groups of the same panels run on the same XCD (workgroup b goes to XCD
// b % 8 and takes unit group b % 8 + 8 j), so a weight tile read by the first
// row group is an L2 hit for the others.
//
// Arithmetic is the skinny engine's, operation for operation: the k-blocks
// of a panel are summed over the same eight k-ranges (range w: k-blocks
// [NKB w / 8, NKB (w + 1) / 8)), each range with a fresh MFMA accumulator in
// the same instruction order, and the range partials are added in range
// order.  A row's result does not depend on the engine or on the other rows.
#pragma once

#include "device_gemm.h"

namespace spade {

constexpr int kWideRowBytes = 256 * 2 + 16;  // one row of one split of a k-block in LDS (+16 B pad)

template <int RT>
struct GemmWideSmem {
  uint8_t ring[2][kActSplits][RT * 16][kWideRowBytes];
  float rinv[RT * 16];
};

template <int RT, int KIND>
struct GemmWide {
  static constexpr int S = kActSplits;
  static constexpr int NST = 2 * RT;  // 16-byte activation chunks per thread and k-block

  const GemmParams& a;
  GemmWideSmem<RT>& sm;
  int tid, lane, wave, g, kl;
  int u;        // this wave's unit
  bool uok;     // the unit exists
  int row0;     // first launch row of the row group
  int NKB, Tpad;
  Rsrc ra[S];
  uint4 w0[8], w1[8], w2[8];
  uint4 st0[NST], st1[NST];
  floatx4 acc[RT], tot[RT];
  int rnext, bnd;  // next k-range index and the k-block its range starts at

  __device__ __forceinline__ GemmWide(const GemmParams& a_, GemmWideSmem<RT>& sm_, int ug, int rg)
      : a(a_), sm(sm_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    g = lane >> 4;
    kl = lane & 15;
    u = ug * kGemmWaves + wave;
    uok = u < a.n_units;
    row0 = rg * RT * 16;
    NKB = a.NKB;
    Tpad = (NKB + 5) / 6 * 6;
#pragma unroll
    for (int s = 0; s < S; ++s)
      ra[s] = make_rsrc((const uint8_t*)a.act + ((size_t)s * a.act_split + (size_t)a.m0 * a.act_stride) * 2,
                        (uint32_t)((size_t)a.M * a.act_stride * 2));
#pragma unroll
    for (int mt = 0; mt < RT; ++mt) {
      acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
      tot[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    rnext = 1;
    bnd = NKB / kGemmWaves;
    while (bnd == 0 && rnext < kGemmWaves) bnd = (NKB * ++rnext) / kGemmWaves;
  }

  // weight tile of k-block kb of this wave's unit (zeros past the panel or
  // for a missing unit)
  __device__ __forceinline__ void issue_w(int kb, uint4 (&w)[8]) const {
    const bool ok = uok && kb < NKB;
    const uint8_t* tile = a.w + ((size_t)(ok ? u : 0) * NKB + (ok ? kb : 0)) * kTileBytes;
    const Rsrc r = make_rsrc(tile, ok ? (uint32_t)kTileBytes : 0u);
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = ld_b128<false>(r, (uint32_t)(lane * 16 + j * 1024));
  }

  // this thread's chunks of activation k-block kb: chunk c = tid + 512 i is
  // (split s, row r, 16-byte column kc); rows past M and k-blocks past NKB
  // read zeros
  __device__ __forceinline__ void issue_a(int kb, uint4 (&st)[NST]) const {
#pragma unroll
    for (int i = 0; i < NST; ++i) {
      const int c = tid + 512 * i;
      const int s = c / (RT * 512), rem = c - s * (RT * 512);
      const int r = rem >> 5, kc = rem & 31;
      const int row = row0 + r;
      const bool ok = row < a.M && kb < NKB;
      const uint32_t off = ok ? (uint32_t)(row * a.act_stride + kb * 256 + kc * 8) * 2u : kOob;
      st[i] = ld_b128<false>(s == 0 ? ra[0] : ra[S - 1], off);
    }
  }

  __device__ __forceinline__ void store_a(int slot, const uint4 (&st)[NST]) {
#pragma unroll
    for (int i = 0; i < NST; ++i) {
      const int c = tid + 512 * i;
      const int s = c / (RT * 512), rem = c - s * (RT * 512);
      const int r = rem >> 5, kc = rem & 31;
      *(uint4*)&sm.ring[slot][s][r][kc * 16] = st[i];
    }
  }

  // MFMAs of one k-block: weights w, activations from ring slot `slot`, in the
  // skinny engine's order (slice j, row tile, split hi before lo... as there:
  // split S-1 first)
  __device__ __forceinline__ void mma(int slot, const uint4 (&w)[8]) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint4 x[RT][S];
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int s = 0; s < S; ++s) x[mt][s] = *(const uint4*)&sm.ring[slot][s][mt * 16 + kl][(32 * j + 8 * g) * 2];
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int s = S - 1; s >= 0; --s)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x[mt][s]),
                                                            __builtin_bit_cast(bf16x8, w[j]), acc[mt], 0, 0, 0);
    }
  }

  // after k-block kb: at the end of a k-range add its partial to the total
  // (ranges in order; an empty range adds nothing, as a zero partial would)
  __device__ __forceinline__ void range_end(int kb) {
    if (kb + 1 == bnd) {
#pragma unroll
      for (int mt = 0; mt < RT; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) tot[mt][i] += acc[mt][i];
        acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
      do {
        ++rnext;
        bnd = (NKB * rnext) / kGemmWaves;
      } while (bnd == kb + 1 && rnext < kGemmWaves);
    }
  }

  // k-block kb: weights in w (refilled with kb + 3), activation block kb + 1
  // in staging set st (written to the ring, refilled with kb + 3)
  __device__ __forceinline__ void step(int kb, uint4 (&w)[8], uint4 (&st)[NST]) {
    __syncthreads();  // block kb visible; the slot of kb - 1 is free
    mma(kb & 1, w);
    __builtin_amdgcn_sched_barrier(0);
    range_end(kb);
    store_a((kb + 1) & 1, st);
    issue_a(kb + 3, st);
    issue_w(kb + 3, w);
  }

  __device__ __forceinline__ void run() {
    // prologue: blocks 0 and 1 of the operand and tiles 0 and 1 (operand
    // first), block 0 into the ring, then block 2 and tile 2
    issue_a(0, st0);
    issue_w(0, w0);
    issue_a(1, st1);
    issue_w(1, w1);
    // row scales of the group while those are in flight
    for (int r = tid >> 4; r < RT * 16; r += 32) {
      const float ri = gemm_row_rinv(a, row0 + r, tid & 15);
      if ((tid & 15) == 0) sm.rinv[r] = ri;
    }
    store_a(0, st0);
    issue_a(2, st0);
    issue_w(2, w2);
    // k-block kb uses weight set kb % 3 and writes staging set (kb + 1) % 2
    for (int kb = 0; kb < Tpad; kb += 6) {
      step(kb, w0, st1);
      step(kb + 1, w1, st0);
      step(kb + 2, w2, st1);
      step(kb + 3, w0, st0);
      step(kb + 4, w1, st1);
      step(kb + 5, w2, st0);
    }
    __syncthreads();  // rinv
    // epilogue: lane holds rows mt*16 + 4g + i, column kl of unit u
#pragma unroll
    for (int mt = 0; mt < RT; ++mt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = mt * 16 + 4 * g + i;
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
        gemm_epilogue<KIND, true, false>(a, uok ? u : 0, ml, kl, rok, pos, bg, sm.rinv[r], tot[mt][i], e);
      }
    }
  }
};

// Host-side shape of a wide launch: row tiles per workgroup and row groups.
inline __host__ __device__ int gemm_wide_row_groups(int M, int rt) { return ((M + 15) / 16 + rt - 1) / rt; }
inline __host__ __device__ uint32_t gemm_wide_lds_bytes(int rt) {
  return (uint32_t)(2 * kActSplits * rt * 16 * kWideRowBytes + rt * 16 * 4);
}

}  // namespace spade
