// Wide-row GEMM for the projections (QKV, O, gate/up, down) and the LM head
// when the activation operand has more rows than the skinny engine
// (device_gemm.h) keeps resident: batched verification, M = B (gamma + 1) up
// to 256 rows.  The LM head stores its logits and, per row and panel, the
// panel's (max, sum exp, argmax); the accept step folds them in the skinny
// engine's order.
//
// A workgroup of 8 waves owns 8P consecutive panels ("units"), P per wave,
// and a group of RT 16-row tiles.  Each wave streams its panels' k-blocks
// (8 KB weight tiles each) through a register pipeline (3 k-blocks deep for
// one panel, 2 for two) and multiplies every tile with all RT row tiles; each
// activation fragment read from LDS feeds P MFMAs.  The activation k-blocks
// (RT * 16 rows x 256 k, two bf16 terms) pass through a three-slot LDS ring
// filled by direct buffer->LDS loads, two k-blocks ahead: right after the
// barrier that ends every wave's reads of the slot k-block kb - 1 used,
// k-block kb + 2 is requested into it, so a fill has two k-blocks of MFMAs to
// land.  Rows of the ring are 512 bytes with their 16-byte chunks
// XOR-swizzled by the row (chunk c of row r holds k-chunk c ^ (r % 16)), so
// the 16 rows of a fragment read hit distinct banks.
//
// The ring is read with inline-asm ds_read_b128 and explicit lgkmcnt waits
// tied to the fragment registers: the compiler, seeing LDS reads while a
// direct-to-LDS load is outstanding, would otherwise wait for every such load
// before the first read and expose each fill's latency.  Each wave instead
// waits (vmcnt) for its own share of k-block kb, then the barrier publishes
// the whole block.
//
// Row groups of the same panels run on the same XCD (workgroup b goes to XCD
// b % 8 and takes unit group b % 8 + 8 j), so a weight tile read by the first
// row group is an L2 hit for the others.
//
// K-splits (KS = 2 or 4; the O and down projections, whose few panels give
// too few workgroups to fill the chip): workgroup split s streams only the
// k-blocks of ranges [8s/KS, 8(s+1)/KS).  Split 0 publishes its running sum
// over its ranges, the other splits each range partial (write-through stores);
// every workgroup then arrives on the counter of its (unit group, row group),
// and the last to arrive continues split 0's sum over the other ranges in
// range order and runs the epilogue.
//
// Arithmetic is the skinny engine's, operation for operation: the k-blocks
// of a panel are summed over the same eight k-ranges (range w: k-blocks
// [NKB w / 8, NKB (w + 1) / 8)), each range with a fresh MFMA accumulator in
// the same instruction order, and the range partials are added in range
// order.  A row's result does not depend on the engine, the tiling or the
// other rows.
#pragma once

#include "device_gemm.h"

#include <utility>

namespace spade {

constexpr int kWideSlots = 3;  // activation ring slots (k-blocks)

template <int RT>
struct GemmWideSmem {
  uint8_t ring[kWideSlots][kActSplits][RT * 16][512];
  float rinv[RT * 16];
  int last;  // k-splits: this workgroup arrived last
};

// Published values of one (unit group, row group) of a k-split launch: slot
// r (0: split 0's running sum, r >= 8/KS: range r), then per wave, panel, row
// tile, accumulator register and lane one float.
template <int RT, int P>
constexpr int kWideItemFloats = 8 * kGemmWaves * P * RT * 256;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// NT: the weight tiles are loaded with the non-temporal policy (launches of
// few row groups, whose tiles are read about once); without it they stay in
// L2 for the other row groups of a many-row launch.
template <int RT, int P, int KIND, int KS = 1, bool NT = true>
struct GemmWide {
  static_assert(KS == 1 || KS == 2 || KS == 4, "k-splits");
  static constexpr int NPR = KS == 2 ? 3 : 1;  // range partials a split > 0 holds besides tot
  static constexpr int S = kActSplits;
  static constexpr int D = P == 1 ? 4 : 2;  // weight pipeline depth in k-blocks
  static constexpr int PERIOD = D == 4 ? 12 : 6;  // lcm(D, kWideSlots): steps per loop iteration
  static constexpr int NFILL = 2 * RT;      // direct LDS loads per wave and k-block
  static_assert(S == 2, "the ring fill gives splits to waves 0-3 and 4-7");

  const GemmParams& a;
  GemmWideSmem<RT>& sm;
  int tid, lane, wave, g, kl;
  int ubase;  // first unit of this wave
  int row0;   // first launch row of the row group
  int NKB;
  int ks, kb0, kb1;  // k-split and its k-blocks [kb0, kb1)
  uint32_t* cnt;     // k-splits: arrival counter of this (unit group, row group)
  float* part;       // k-splits: its published values (kWideItemFloats)
  Rsrc rfill;  // this wave's split of the operand
  uint32_t lds_ring;  // LDS byte address of the ring
  uint32_t aoff[4];   // this lane's fragment offsets within a slot (slice j: aoff[j % 4] + 256 (j / 4))
  uint4 wset[D][P][8];
  floatx4 acc[RT][P], tot[RT][P];
  floatx4 pr[NPR][RT][P];  // split > 0: earlier range partials, latest first
  int rnext, bnd;  // next k-range index and the k-block its range starts at

  __device__ __forceinline__ GemmWide(const GemmParams& a_, GemmWideSmem<RT>& sm_, int ug, int rg, int ks_ = 0,
                                      uint32_t* cnt_ = nullptr, float* part_ = nullptr)
      : a(a_), sm(sm_), ks(ks_), cnt(cnt_), part(part_) {
    tid = threadIdx.x;
    lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    g = lane >> 4;
    kl = lane & 15;
    ubase = (ug * kGemmWaves + wave) * P;
    row0 = rg * RT * 16;
    NKB = a.NKB;
    lds_ring = (uint32_t)(size_t)(__attribute__((address_space(3))) void*)&sm.ring[0][0][0][0];
#pragma unroll
    for (int t = 0; t < 4; ++t) aoff[t] = (uint32_t)(kl * 512 + 64 * (t ^ (kl >> 2)) + 16 * (g ^ (kl & 3)));
    const int s = wave >> 2;
    rfill = make_rsrc((const uint8_t*)a.act + ((size_t)s * a.act_split + (size_t)a.m0 * a.act_stride) * 2,
                      (uint32_t)((size_t)a.M * a.act_stride * 2));
#pragma unroll
    for (int mt = 0; mt < RT; ++mt)
#pragma unroll
      for (int p = 0; p < P; ++p) {
        acc[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
        tot[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < NPR; ++q) pr[q][mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
    // ranges [r_lo, r_hi) of this split; rnext / bnd: the first non-empty one
    const int r_lo = kGemmWaves * ks / KS, r_hi = kGemmWaves * (ks + 1) / KS;
    kb0 = NKB * r_lo / kGemmWaves;
    kb1 = NKB * r_hi / kGemmWaves;
    rnext = r_lo + 1;
    bnd = NKB * rnext / kGemmWaves;
    while (bnd == kb0 && rnext < r_hi) bnd = (NKB * ++rnext) / kGemmWaves;
  }

  // weight tiles of k-block kb of this wave's units (zeros past the panel or
  // for a missing unit)
  __device__ __forceinline__ void issue_w(int kb, uint4 (&w)[P][8]) const {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int u = ubase + p;
      const bool ok = u < a.n_units && kb < kb1;
      const uint8_t* tile = a.w + ((size_t)(ok ? u : 0) * NKB + (ok ? kb : 0)) * kTileBytes;
      const Rsrc r = make_rsrc(tile, ok ? (uint32_t)kTileBytes : 0u);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if constexpr (NT) w[p][j] = ld_stream_b128(r, (uint32_t)(lane * 16 + j * 1024));
        else w[p][j] = ld_b128<false>(r, (uint32_t)(lane * 16 + j * 1024));
      }
    }
  }

  // Request activation k-block kb into ring slot `slot`.  Waves 0-3 move
  // split 0 and waves 4-7 split 1; one load instruction moves two rows (lane
  // l: row 2 rp + l / 32, LDS chunk l % 32).  Rows past M repeat row M - 1:
  // finite values whose products are never stored.  K-blocks past this
  // split's end read nothing (the loop never reaches them).
  __device__ __forceinline__ void fill(int kb, int slot) const {
    const int s = wave >> 2;
    const bool kok = kb < kb1;
    const int c = lane & 31;
#pragma unroll
    for (int i = 0; i < NFILL; ++i) {
      const int rp = (wave & 3) + 4 * i;
      const int row = 2 * rp + (lane >> 5);
      const int grow = row0 + row < a.M ? row0 + row : a.M - 1;
      const int gc = c ^ (row & 15);
      const uint32_t off = kok ? (uint32_t)(grow * a.act_stride + kb * 256 + gc * 8) * 2u : kOob;
      __attribute__((address_space(3))) void* dst =
          (__attribute__((address_space(3))) void*)&sm.ring[slot][s][2 * rp][0];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rfill, dst, 16, off, 0, 0, 0);
    }
  }

  // 16-byte ring read at LDS byte address addr + OFF (inline asm: the
  // compiler neither sees the LDS access nor waits for it)
  template <int OFF>
  __device__ __forceinline__ static u32x4 ds_read16(uint32_t addr) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
  }

  // wait until at most N LDS reads are outstanding, ordered before every use
  // of the fragments x
  template <int N>
  __device__ __forceinline__ static void lds_wait(u32x4 (&x)[RT][S]) {
#pragma unroll
    for (int mt = 0; mt < RT; ++mt)
#pragma unroll
      for (int s = 0; s < S; ++s) asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x[mt][s]) : "n"(N));
  }

  // fragments of slice j (row tile mt, split s) from the ring slot whose
  // per-lane base addresses are ab[t], t = j % 4
  template <int J, int... I>
  __device__ __forceinline__ static void read_slice_i(const uint32_t (&ab)[4], u32x4 (&x)[RT][S],
                                                      std::integer_sequence<int, I...>) {
    // I = s * RT + mt
    ((x[I % RT][I / RT] = ds_read16<I * 16 * 512 + 256 * (J >> 2)>(ab[J & 3])), ...);
  }
  template <int J>
  __device__ __forceinline__ static void read_slice(const uint32_t (&ab)[4], u32x4 (&x)[RT][S]) {
    read_slice_i<J>(ab, x, std::make_integer_sequence<int, RT * S>{});
  }

  template <int J>
  __device__ __forceinline__ void mma_slice(const u32x4 (&x)[RT][S], const uint4 (&w)[P][8]) {
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int s = S - 1; s >= 0; --s)
          acc[mt][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x[mt][s]),
                                                               __builtin_bit_cast(bf16x8, w[p][J]), acc[mt][p], 0, 0, 0);
  }

  // MFMAs of one k-block: weights w, activations from ring slot `slot`, for
  // every accumulator in the skinny engine's order (slice j, split S-1 first).
  // Fragment reads run one slice ahead of the MFMAs.  Chunk (4j + g) ^ kl of
  // row kl sits at byte 256 (j / 4) + 64 ((j % 4) ^ (kl / 4)) + 16 (g ^ kl % 4).
  __device__ __forceinline__ void mma(int slot, const uint4 (&w)[P][8]) {
    const uint32_t sb = lds_ring + (uint32_t)slot * (uint32_t)(kActSplits * RT * 16 * 512);
    uint32_t ab[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) ab[t] = sb + aoff[t];
    u32x4 xa[RT][S], xb[RT][S];
    read_slice<0>(ab, xa);
    read_slice<1>(ab, xb);
    lds_wait<RT * S>(xa);
    mma_slice<0>(xa, w);
    read_slice<2>(ab, xa);
    lds_wait<RT * S>(xb);
    mma_slice<1>(xb, w);
    read_slice<3>(ab, xb);
    lds_wait<RT * S>(xa);
    mma_slice<2>(xa, w);
    read_slice<4>(ab, xa);
    lds_wait<RT * S>(xb);
    mma_slice<3>(xb, w);
    read_slice<5>(ab, xb);
    lds_wait<RT * S>(xa);
    mma_slice<4>(xa, w);
    read_slice<6>(ab, xa);
    lds_wait<RT * S>(xb);
    mma_slice<5>(xb, w);
    read_slice<7>(ab, xb);
    lds_wait<RT * S>(xa);
    mma_slice<6>(xa, w);
    lds_wait<0>(xb);
    mma_slice<7>(xb, w);
  }

  // after k-block kb: at the end of a k-range add its partial to the total
  // (ranges in order; an empty range adds nothing, as a zero partial would).
  // A k-split other than the first keeps each range partial instead: the
  // latest in tot, the earlier ones in pr (latest first).
  __device__ __forceinline__ void range_end(int kb) {
    if (kb + 1 == bnd) {
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int p = 0; p < P; ++p) {
          if (KS == 1 || ks == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) tot[mt][p][i] += acc[mt][p][i];
          } else {
#pragma unroll
            for (int q = NPR - 1; q > 0; --q) pr[q][mt][p] = pr[q - 1][mt][p];
            pr[0][mt][p] = tot[mt][p];
            tot[mt][p] = acc[mt][p];
          }
          acc[mt][p] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
      do {
        ++rnext;
        bnd = (NKB * rnext) / kGemmWaves;
      } while (bnd == kb + 1 && rnext < kGemmWaves);
    }
  }

  // k-block kb: weights in set WS (refilled with kb + D), activations in ring
  // slot SLOT = kb % 3.  On entry the vector-memory operations issued after
  // the fill of kb are at most the weights of two steps and one fill (steady
  // state; fewer in the first steps), so waiting for that count completes this
  // wave's share of k-block kb; the barrier then publishes every wave's share
  // and ends the reads of slot (kb + 2) % 3, into which k-block kb + 2 is
  // requested.  The barrier is a bare s_barrier: the ring is read with inline
  // asm and written by direct loads whose completion each wave has just
  // waited for, so no fence is needed (a workgroup fence would also wait for
  // the fill of kb + 1 and everything issued before it, draining the weight
  // pipeline).
  template <int SLOT, int WS>
  __device__ __forceinline__ void step(int kb) {
    wait_vmcnt<NFILL + 16 * P>();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    fill(kb + 2, (SLOT + 2) % kWideSlots);
    mma(SLOT, wset[WS]);
    __builtin_amdgcn_sched_barrier(0);
    range_end(kb);
    issue_w(kb + D, wset[WS]);
  }

  template <int... I>
  __device__ __forceinline__ void period_steps(int kb, std::integer_sequence<int, I...>) {
    (step<I % kWideSlots, I % D>(kb + I), ...);
  }

  // the first n (< PERIOD) steps of a period, n uniform
  template <int... I>
  __device__ __forceinline__ void tail_steps(int kb, int n, std::integer_sequence<int, I...>) {
    ((I < n ? step<I % kWideSlots, I % D>(kb + I) : void()), ...);
  }

  // Byte offset of (slot, panel p, row tile mt, register i) of this lane in
  // the published values of a k-split launch.
  __device__ __forceinline__ uint32_t part_off(int slot, int p, int mt, int i) const {
    return (uint32_t)(((((slot * kGemmWaves + wave) * P + p) * RT + mt) * 4 + i) * 64 + lane) * 4u;
  }

  // K-splits: publish this split's values, arrive, and in the last workgroup
  // to arrive leave in tot the full sums (split 0's running sum, then the
  // non-empty ranges of the other splits in range order).  Returns whether
  // this workgroup runs the epilogue (uniform).
  __device__ __forceinline__ bool combine_splits() {
    const Rsrc rp = make_rsrc(part, (uint32_t)kWideItemFloats<RT, P> * 4u);
    const int r_lo = kGemmWaves * ks / KS, r_hi = kGemmWaves * (ks + 1) / KS;
    auto nonempty = [&](int r) { return NKB * (r + 1) / kGemmWaves > NKB * r / kGemmWaves; };
    // value q (tot, then pr[q - 1]) holds the q-th non-empty range from the
    // top of this split; split 0 stores only its running sum, in slot 0
    int slot[NPR + 1];
    {
      int q = 0;
#pragma unroll
      for (int i = 0; i <= NPR; ++i) slot[i] = -1;
      for (int r = r_hi - 1; r >= r_lo; --r)
        if (nonempty(r)) {
#pragma unroll
          for (int i = 0; i <= NPR; ++i)
            if (i == q) slot[i] = r;
          ++q;
        }
      if (ks == 0) {
        slot[0] = 0;
#pragma unroll
        for (int i = 1; i <= NPR; ++i) slot[i] = -1;
      }
    }
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          st_f32<true>(rp, slot[0] >= 0 ? part_off(slot[0], p, mt, i) : kOob, tot[mt][p][i]);
#pragma unroll
          for (int q = 1; q <= NPR; ++q)
            st_f32<true>(rp, slot[q] >= 0 ? part_off(slot[q], p, mt, i) : kOob, pr[q - 1][mt][p][i]);
        }
    // every published value has landed: arrive
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
      const uint32_t old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int last = old == (uint32_t)KS - 1u;
      if (last) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      sm.last = last;
    }
    __syncthreads();
    if (!sm.last) return false;
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v[kGemmWaves];
#pragma unroll
          for (int r = 0; r < kGemmWaves; ++r) {
            const bool use = r == 0 || (r >= kGemmWaves / KS && nonempty(r));
            v[r] = ld_b32_coh(rp, use ? part_off(r, p, mt, i) : kOob);
          }
          float t = v[0];
#pragma unroll
          for (int r = kGemmWaves / KS; r < kGemmWaves; ++r)
            if (nonempty(r)) t += v[r];
          tot[mt][p][i] = t;
        }
    return true;
  }

  __device__ __forceinline__ void run() {
    // prologue: the split's first two k-blocks of the operand, the first D
    // weight sets
    fill(kb0, 0);
    fill(kb0 + 1, 1);
    // the fills stay older than every weight load (the waits count on it)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < D; ++i) issue_w(kb0 + i, wset[i]);
    // whole periods in a loop (no exits inside, so the compiler's wait counts
    // at the loop head stay exact), then the remaining k-blocks
    const int n = kb1 - kb0;
    const int full = n / PERIOD * PERIOD;
    for (int t = 0; t < full; t += PERIOD) period_steps(kb0 + t, std::make_integer_sequence<int, PERIOD>{});
    tail_steps(kb0 + full, n - full, std::make_integer_sequence<int, PERIOD - 1>{});
    // the last fills (k-blocks past the end) must land before the ring is
    // reused; the row scales are only needed by the epilogue
    __builtin_amdgcn_s_waitcnt(0);
    for (int r = tid >> 4; r < RT * 16; r += 32) {
      const float ri = gemm_row_rinv(a, row0 + r, tid & 15);
      if ((tid & 15) == 0) sm.rinv[r] = ri;
    }
    __syncthreads();
    if constexpr (KS > 1)
      if (!combine_splits()) return;
    // epilogue: lane holds rows mt*16 + 4g + i, column kl of each unit
    bool nan_seen = false;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int u = ubase + p;
      const bool uok = u < a.n_units;
#pragma unroll
      for (int mt = 0; mt < RT; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = mt * 16 + 4 * g + i;
          const int ml = row0 + r;
          const bool rok = uok && ml < a.M;
          if constexpr (KIND == GEMM_LM) {
            // logits and the panel's statistics (the accept step folds the
            // panels in the skinny engine's workgroup order)
            const bool samp = gemm_lm_samp(a, ml, rok);
            const RowStat ps =
                gemm_lm_panel<false>(a, uok ? u : 0, ml, kl, rok, samp, sm.rinv[r], tot[mt][p][i], nan_seen);
            gemm_lm_store_panel(a, uok ? u : 0, ml, kl, rok, ps);
          } else {
            int pos = 0, bg = 0;
            if constexpr (KIND == GEMM_QKV) {
              const int m = a.m0 + ml;
              const int bl = m / a.R, ir = m - bl * a.R;
              bg = a.b0 + bl;
              if (rok) pos = a.lens[bg] + ir;
            }
            const EpiIn e = gemm_epi_load<KIND, false>(a, uok ? u : 0, ml, kl, rok, pos);
            gemm_epilogue<KIND, true, false>(a, uok ? u : 0, ml, kl, rok, pos, bg, sm.rinv[r], tot[mt][p][i], e);
          }
        }
      }
    }
    if (nan_seen) flag_error(a.err, SPADE_DERR_NAN);
  }
};

// Host-side shape of a wide launch.
inline __host__ __device__ int gemm_wide_row_groups(int M, int rt) { return ((M + 15) / 16 + rt - 1) / rt; }
inline __host__ __device__ int gemm_wide_unit_groups(int n_units, int p) {
  return (n_units + kGemmWaves * p - 1) / (kGemmWaves * p);
}
inline __host__ __device__ uint32_t gemm_wide_lds_bytes(int rt) {
  return (uint32_t)(kWideSlots * kActSplits * rt * 16 * 512 + rt * 16 * 4 + 16);
}

}  // namespace spade
