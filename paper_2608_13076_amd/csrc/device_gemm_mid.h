// GEMM for the projections of batched verification with up to 144 rows
// (QKV, O, gate/up and down; M = B (gamma + 1), e.g. 16 requests of 9 rows):
// every row of the call in one workgroup, so each weight byte enters one
// compute unit once per launch.
//
// A workgroup of 8 waves (two per SIMD) owns all kMidRT row tiles and 16
// panels (256 columns); wave w takes panels 2w and 2w + 1 with every row
// tile: 18 MFMA output tiles, each with a running k-range accumulator and a
// total.  The k-loop runs in 32-k slices (one MFMA k-step, 8 per 256-k
// block).  A slice of the activations (144 rows x 32 k x two bf16 terms,
// 18 KB) goes by direct buffer->LDS loads into a five-slot ring, four slices
// ahead; each wave reads every row tile's fragments (inline-asm ds_read_b128
// with explicit waits), each feeding 2 MFMAs.  The weight fragments of a
// slice (1 KB per panel) load straight into a four-slice register ring.
//
// The gate/up projection of a 7B model at 144 rows has 86 such panel groups,
// its O and down projections 16: K-splits fill the chip.  Workgroup (panel
// group, split s of KS) streams the k-blocks of k-ranges [8s/KS, 8(s+1)/KS);
// split 0 keeps a running total over its ranges and stores it at the end,
// every other split stores each range partial as soon as the range ends
// (write-through).  A second launch (gemm_mid_finish_kernel), one workgroup
// per panel group and row tile, adds the other splits' range partials to
// split 0's total in range order and runs the epilogue: the published values
// (147 KB per slot and panel group) are read by hundreds of compute units at
// once instead of by one per panel group.
//
// Arithmetic is the skinny engine's, operation for operation: per output,
// the k-blocks of each of the eight k-ranges (range r: k-blocks
// [NKB r / 8, NKB (r + 1) / 8)) accumulate in a fresh MFMA accumulator, slice
// by slice, the low bf16 term of the activation before the high one; the
// range partials are added to the total in range order (an empty range adds
// nothing).  A row's result does not depend on the engine, the k-splits or
// the other rows.
#pragma once

#include "device_gemm.h"

#include <utility>

namespace spade {

constexpr int kMidWaves = 8;
constexpr int kMidRT = 9;                          // row tiles per workgroup (144 rows)
constexpr int kMidP = 2;                           // panels per wave
constexpr int kMidUnits = kMidWaves * kMidP;       // panels per workgroup
constexpr int kMidSlots = 5;                       // activation slices in the LDS ring
constexpr int kMidDepth = 4;                       // slices requested ahead (divides the 8 of a k-block)
constexpr int kMidBlocks = kActSplits * kMidRT;    // 1 KB (split, row tile) blocks per slice
constexpr int kMidMaxSplits = 8;

// Published values of one panel group: slot r (0: split 0's total, else
// range r's partial), then per wave, panel, row tile and lane one floatx4.
constexpr int kMidItemFloats = 8 * kMidWaves * kMidP * kMidRT * 64 * 4;

struct GemmMidSmem {
  // slot, split, row tile: 16 rows x 64 bytes, the four 16-byte pieces of row
  // r at piece p ^ f(r), f(r) = ((r / 2) ^ (r / 4)) % 4 (the rows of a
  // fragment read that share a pass land on distinct banks)
  uint8_t ring[kMidSlots][kActSplits][kMidRT][1024];
  uint8_t pad[1024];  // target of the fill loads past the 18 blocks (never read)
};

typedef uint32_t u32x4m __attribute__((ext_vector_type(4)));

template <int KIND>
struct GemmMid {
  static_assert(KIND != GEMM_LM, "projections only");
  static constexpr int S = kActSplits;
  static constexpr int D = kMidDepth;
  static constexpr int RT = kMidRT;
  static constexpr int P = kMidP;
  static constexpr int NF = (kMidBlocks + kMidWaves - 1) / kMidWaves;  // fill loads per wave and slice
  static_assert(NF == 3, "fill: three loads per wave and slice");
  static_assert(8 % D == 0, "the weight ring is indexed by the slice within its k-block");
  const GemmParams& a;
  GemmMidSmem& sm;
  int tid, lane, wave, g, kl;
  int u0;              // first panel of this wave
  int NKB, ks, KS;     // k-blocks of the projection; this k-split of KS
  int kb0, kb1, T;     // k-blocks [kb0, kb1) of the split, T = 8 (kb1 - kb0) slices
  float* part;         // published values of the panel group (kMidItemFloats)
  uint32_t lds_ring;   // LDS byte address of the ring
  uint32_t frag_off;   // this lane's fragment offset within a 1 KB block
  uint32_t foff[3];    // this lane's byte offsets of its fill blocks at k 0 (past the resource: none)
  Rsrc ract;           // activations of the launch's rows, both splits
  Rsrc rw[P];          // this wave's weight panels (empty past n_units)
  Rsrc rp;             // published values of the panel group
  floatx4 acc[RT][P], tot[RT][P];
  uint4 wq[D][P];      // weight fragments of the slices in flight
  int rnext, bnd;      // next k-range, the k-block its range starts at

  __device__ __forceinline__ GemmMid(const GemmParams& a_, GemmMidSmem& sm_, int ug, int ks_, int KS_, float* part_)
      : a(a_), sm(sm_), ks(ks_), KS(KS_), part(part_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    g = lane >> 4;
    kl = lane & 15;
    u0 = ug * kMidUnits + wave * P;
    NKB = a.NKB;
    lds_ring = (uint32_t)(size_t)(__attribute__((address_space(3))) void*)&sm.ring[0][0][0][0];
    frag_off = (uint32_t)(kl * 64 + 16 * (g ^ (((kl >> 1) ^ (kl >> 2)) & 3)));
    ract = make_rsrc((const uint8_t*)a.act + (size_t)a.m0 * a.act_stride * 2,
                     (uint32_t)(((size_t)(S - 1) * a.act_split + (size_t)a.M * a.act_stride) * 2));
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int u = u0 + p;
      const bool ok = u < a.n_units;
      rw[p] = make_rsrc(a.w + (size_t)(ok ? u : 0) * NKB * kTileBytes, ok ? (uint32_t)(NKB * kTileBytes) : 0u);
    }
    rp = make_rsrc(part, (uint32_t)kMidItemFloats * 4u);
#pragma unroll
    for (int mt = 0; mt < RT; ++mt)
#pragma unroll
      for (int p = 0; p < P; ++p) {
        acc[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
        tot[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
    // ranges [r_lo, r_hi) of this split; rnext / bnd: the first non-empty one
    const int r_lo = kGemmWaves * ks / KS, r_hi = kGemmWaves * (ks + 1) / KS;
    kb0 = NKB * r_lo / kGemmWaves;
    kb1 = NKB * r_hi / kGemmWaves;
    T = (kb1 - kb0) * 8;
    rnext = r_lo + 1;
    bnd = NKB * rnext / kGemmWaves;
    while (bnd == kb0 && rnext < r_hi) bnd = (NKB * ++rnext) / kGemmWaves;
    // fill offsets at the split's first k-block
    {
      const int r = lane >> 2, pp = lane & 3;
      const int lp = pp ^ (((r >> 1) ^ (r >> 2)) & 3);
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int q = wave + kMidWaves * i;
        const int s = q / RT, mt = q - s * RT;
        const int row = mt * 16 + r;
        const int grow = row < a.M ? row : a.M - 1;
        foff[i] = q < kMidBlocks
                      ? (uint32_t)(((size_t)s * a.act_split + (size_t)grow * a.act_stride + (size_t)kb0 * 256 + lp * 8) * 2)
                      : kOob;
      }
    }
  }

  // Request slice t of the split (its k-block kb0 + t / 8, k-step t % 8) into
  // ring slot t % kMidSlots: wave w moves blocks w, w + 8 and w + 16 of the
  // 18 (split, row tile) blocks, one 16-byte piece per lane (lane l: row
  // l / 4, piece l % 4 of the swizzled block); waves 2-7 have no third block
  // and read nothing (an offset past the resource) into the pad, so every
  // wave issues the same loads and the wait counts are the same constants.
  // Rows past M repeat row M - 1: finite values whose products are never
  // stored.  Slices past the split read zeros into a slot no later slice
  // reads.
  __device__ __forceinline__ void fill(int t) const {
    const int slot = t % kMidSlots;
    const uint32_t kofs = (uint32_t)(((t >> 3) * 256 + (t & 7) * 32) * 2);
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int q = wave + kMidWaves * i;
      const bool real = q < kMidBlocks;
      const int s = q / RT, mt = q - s * RT;
      const uint32_t off = t < T ? foff[i] + kofs : kOob;
      __attribute__((address_space(3))) void* dst =
          real ? (__attribute__((address_space(3))) void*)&sm.ring[slot][real ? s : 0][real ? mt : 0][0]
               : (__attribute__((address_space(3))) void*)&sm.pad[0];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ract, dst, 16, off, 0, 0, 0);
    }
  }

  // weight fragments of slice t for this wave's panels (zeros past the
  // split: the offset is past the resource)
  __device__ __forceinline__ void issue_w(int t, uint4 (&w)[P]) const {
    const uint32_t off = t < T ? (uint32_t)((kb0 + (t >> 3)) * kTileBytes + (t & 7) * 1024 + lane * 16) : kOob;
#pragma unroll
    for (int p = 0; p < P; ++p) w[p] = ld_stream_b128(rw[p], off);
  }

  template <int OFF>
  __device__ __forceinline__ static u32x4m ds_read16(uint32_t addr) {
    u32x4m v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
  }

  // fragments of row tiles MT0 .. MT0 + 2 (both splits) into x
  template <int MT0>
  __device__ __forceinline__ static void read3(uint32_t base, u32x4m (&x)[3][S]) {
    x[0][0] = ds_read16<MT0 * 1024>(base);
    x[0][1] = ds_read16<RT * 1024 + MT0 * 1024>(base);
    x[1][0] = ds_read16<(MT0 + 1) * 1024>(base);
    x[1][1] = ds_read16<RT * 1024 + (MT0 + 1) * 1024>(base);
    x[2][0] = ds_read16<(MT0 + 2) * 1024>(base);
    x[2][1] = ds_read16<RT * 1024 + (MT0 + 2) * 1024>(base);
  }

  // wait until at most N of this wave's LDS reads are outstanding; the
  // fragments x depend on the wait
  template <int N>
  __device__ __forceinline__ static void lds_wait_n(u32x4m (&x)[S]) {
#pragma unroll
    for (int s = 0; s < S; ++s) asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x[s]) : "n"(N));
  }

  __device__ __forceinline__ void mma_tile(int mt, const u32x4m (&x)[S], const uint4 (&w)[P]) {
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int s = S - 1; s >= 0; --s)
        acc[mt][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x[s]),
                                                             __builtin_bit_cast(bf16x8, w[p]), acc[mt][p], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);  // keep the tile's MFMAs before the next wait
  }

  // The MFMAs of slice t: fragments of its ring slot, weights w.  Row tiles
  // 0-2 and 3-5 are requested first (12 reads); once 0-2 have gone through
  // the MFMAs, 6-8 are requested into their registers.  LDS reads complete in
  // order, so each row tile starts once at most the reads after its own are
  // outstanding.
  __device__ __forceinline__ void mma(int t, const uint4 (&w)[P]) {
    const uint32_t base = lds_ring + (uint32_t)(t % kMidSlots) * (uint32_t)(S * RT * 1024) + frag_off;
    u32x4m xa[3][S], xb[3][S];
    read3<0>(base, xa);
    read3<3>(base, xb);
    lds_wait_n<10>(xa[0]);
    mma_tile(0, xa[0], w);
    lds_wait_n<8>(xa[1]);
    mma_tile(1, xa[1], w);
    lds_wait_n<6>(xa[2]);
    mma_tile(2, xa[2], w);
    read3<6>(base, xa);
    lds_wait_n<10>(xb[0]);
    mma_tile(3, xb[0], w);
    lds_wait_n<8>(xb[1]);
    mma_tile(4, xb[1], w);
    lds_wait_n<6>(xb[2]);
    mma_tile(5, xb[2], w);
    lds_wait_n<4>(xa[0]);
    mma_tile(6, xa[0], w);
    lds_wait_n<2>(xa[1]);
    mma_tile(7, xa[1], w);
    lds_wait_n<0>(xa[2]);
    mma_tile(8, xa[2], w);
  }

  // Byte offset of (slot, panel p, row tile mt) of this lane in the
  // published values.
  __device__ __forceinline__ uint32_t part_off(int slot, int p, int mt) const {
    return (uint32_t)((((slot * kMidWaves + wave) * P + p) * RT + mt) * 64 + lane) * 16u;
  }

  __device__ __forceinline__ void st4(uint32_t off, const floatx4& v) const {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4m, v), rp, (int)off, 0, kAuxCoh);
  }

  // After k-block kb: at the end of a k-range split 0 adds the range's
  // partial to its total (ranges in order), another split stores it in the
  // range's slot of the published values; the accumulators start the next
  // range at zero.
  __device__ __forceinline__ void range_end(int kb) {
    if (kb + 1 == bnd) {
      if (ks != 0) {
        // (p, mt) of a slot are 1 KB apart
        const uint32_t sbase = part_off(rnext - 1, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mt = 0; mt < RT; ++mt)
#pragma unroll
          for (int p = 0; p < P; ++p) st4(sbase + (uint32_t)((p * RT + mt) * 1024), acc[mt][p]);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int p = 0; p < P; ++p) {
          if (ks == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) tot[mt][p][i] += acc[mt][p][i];
          }
          acc[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
      do {
        ++rnext;
        bnd = (NKB * rnext) / kGemmWaves;
      } while (bnd == kb + 1 && rnext < kGemmWaves);
    }
  }

  // Wait for this wave's share of slice t's fill and for its weights: loads
  // complete in issue order, and the D - 1 slices after slice t have
  // (fills + weights) loads each, so at most that many outstanding operations
  // leaves slice t's loads done.  Stores of published partials may complete
  // out of order with the loads: counted or not, they only make the wait
  // stricter.
  __device__ __forceinline__ static void wait_slice() { wait_vmcnt<(D - 1) * (NF + P)>(); }

  // slice t = 8 (kb - kb0) + J: wait, publish the slot to every wave (bare
  // barrier: the ring is read with inline asm and written by direct loads
  // each wave has waited for), request slice t + D into slot
  // (t + D) % kMidSlots -- the slot of slice t - 1, which every wave finished
  // reading before this barrier -- then the MFMAs, then the weights of slice
  // t + D into the registers just used.
  template <int J>
  __device__ __forceinline__ void slice(int t) {
    wait_slice();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    fill(t + D);
    mma(t, wq[J % D]);
    __builtin_amdgcn_sched_barrier(0);
    issue_w(t + D, wq[J % D]);
  }

  template <int... I>
  __device__ __forceinline__ void kblock(int t0, std::integer_sequence<int, I...>) {
    (slice<I>(t0 + I), ...);
  }

  __device__ __forceinline__ void run() {
    // prologue: the first D slices (each its fill, then its weights: the
    // waits count them in that order)
#pragma unroll
    for (int i = 0; i < D; ++i) {
      fill(i);
      issue_w(i, wq[i]);
    }
    for (int kb = kb0; kb < kb1; ++kb) {
      kblock((kb - kb0) * 8, std::make_integer_sequence<int, 8>{});
      range_end(kb);
    }
    // split 0 publishes its total (the other splits' range partials are
    // out); the workgroup ends once the fills past the split have landed in
    // its LDS
    if (ks == 0) {
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int p = 0; p < P; ++p) st4(part_off(0, p, mt), tot[mt][p]);
    }
    __builtin_amdgcn_s_waitcnt(0);
  }
};

// Second pass of a medium-M launch: workgroup (panel group ug, row tile mt),
// wave w the panels 2w and 2w + 1 of the group as in the first pass, lane l
// the MFMA output layout (column l % 16, rows 4 (l / 16) .. + 3).  Each
// output's sum is split 0's total plus the non-empty ranges of the other
// splits in range order; then the projection's epilogue.
template <int KIND>
struct GemmMidFinish {
  const GemmParams& a;
  float* rinv;  // LDS: 1/rms of the tile's 16 rows
  int tid, lane, wave, g, kl, ug, mt, KS;
  Rsrc rp;

  __device__ __forceinline__ GemmMidFinish(const GemmParams& a_, float* rinv_, int ug_, int mt_, int KS_,
                                           const float* part)
      : a(a_), rinv(rinv_), ug(ug_), mt(mt_), KS(KS_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    g = lane >> 4;
    kl = lane & 15;
    rp = make_rsrc(part + (size_t)ug * kMidItemFloats, (uint32_t)kMidItemFloats * 4u);
  }

  __device__ __forceinline__ uint32_t off(int slot, int p) const {
    return (uint32_t)((((slot * kMidWaves + wave) * kMidP + p) * kMidRT + mt) * 64 + lane) * 16u;
  }

  __device__ __forceinline__ void run() {
    // row scales of the tile's rows (16 threads a row), while the sums load
    if (tid < 256) {
      const float ri = gemm_row_rinv(a, mt * 16 + (tid >> 4), tid & 15);
      if ((tid & 15) == 0) rinv[tid >> 4] = ri;
    }
    const int NKB = a.NKB;
    floatx4 v[kMidP];
#pragma unroll
    for (int p = 0; p < kMidP; ++p) v[p] = __builtin_bit_cast(floatx4, ld_b128<true>(rp, off(0, p)));
    floatx4 x[kGemmWaves - 1][kMidP];
#pragma unroll
    for (int r = 1; r < kGemmWaves; ++r) {
      const bool use = r >= kGemmWaves / KS && NKB * (r + 1) / kGemmWaves > NKB * r / kGemmWaves;
#pragma unroll
      for (int p = 0; p < kMidP; ++p)
        x[r - 1][p] = __builtin_bit_cast(floatx4, ld_b128<true>(rp, use ? off(r, p) : kOob));
    }
#pragma unroll
    for (int r = 1; r < kGemmWaves; ++r) {
      const bool use = r >= kGemmWaves / KS && NKB * (r + 1) / kGemmWaves > NKB * r / kGemmWaves;
      if (use) {
#pragma unroll
        for (int p = 0; p < kMidP; ++p)
#pragma unroll
          for (int i = 0; i < 4; ++i) v[p][i] += x[r - 1][p][i];
      }
    }
    __syncthreads();
    // epilogue: the inputs of the lane's 8 outputs first, then the outputs
    EpiIn e[kMidP][4];
    int pos[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = mt * 16 + 4 * g + i;
      pos[i] = 0;
      if constexpr (KIND == GEMM_QKV) {
        const int m = a.m0 + r;
        const int bl = m / a.R, ir = m - bl * a.R;
        if (r < a.M) pos[i] = a.lens[a.b0 + bl] + ir;
      }
    }
#pragma unroll
    for (int p = 0; p < kMidP; ++p) {
      const int u = ug * kMidUnits + wave * kMidP + p;
      const bool uok = u < a.n_units;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = mt * 16 + 4 * g + i;
        e[p][i] = gemm_epi_load<KIND, false>(a, uok ? u : 0, r, kl, uok && r < a.M, pos[i]);
      }
    }
#pragma unroll
    for (int p = 0; p < kMidP; ++p) {
      const int u = ug * kMidUnits + wave * kMidP + p;
      const bool uok = u < a.n_units;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = mt * 16 + 4 * g + i;
        const int bg = KIND == GEMM_QKV ? a.b0 + (a.m0 + r) / a.R : 0;
        gemm_epilogue<KIND, true, false>(a, uok ? u : 0, r, kl, uok && r < a.M, pos[i], bg, rinv[4 * g + i],
                                         v[p][i], e[p][i]);
      }
    }
  }
};

// Host-side shape of a launch: panel groups; workgroups = groups x k-splits.
inline __host__ __device__ int gemm_mid_unit_groups(int n_units) { return (n_units + kMidUnits - 1) / kMidUnits; }

}  // namespace spade
