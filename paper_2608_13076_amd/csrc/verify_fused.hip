// The verify pass of SPADE's cloud verifier (Algorithm 1, Cloud step; Sec.
// III-A and III-C) as ONE persistent cooperative launch on gfx950.
//
// One 8-wave workgroup per compute unit walks the stages
//   embed | per layer: QKV, attention, O, gate/up, down | LM head | accept
// separated by grid barriers.  The same arithmetic as the per-stage kernels
// (device_gemm.h, device_accept.h; the attention below follows the split-key
// attention of kernels.hip), but
//   * nothing waits for a kernel boundary: a workgroup that reaches a barrier
//     first requests the weight tiles of its first three items of the next
//     stage (they do not depend on anything the current stage writes) and
//     only then waits, so HBM keeps streaming through the barrier; before the
//     attention barrier it requests the cached K/V rows older than this call;
//   * the barrier is split-phase and fence-free: every wave waits for its own
//     stores to complete (s_waitcnt), one thread adds 1 to the counter of its
//     XCD group (blockIdx % 8), and the waiting wave polls the eight group
//     counters with one load per lane;
//   * data one workgroup writes and another reads in the same launch is
//     stored write-through (sc1).  The activations of every stage live in a
//     region of their own per layer (FusedArena), so no L2 holds a line of
//     them before it is written and readers use plain cached loads; the
//     residual stream, the attention partials and the new K/V rows (a line of
//     which an older-row prefetch may already have cached) are read with sc1
//     loads;
//   * the chunk partials of one (request, head) are merged by the last
//     workgroup to finish a chunk (an arrival counter per (request, head)),
//     not by a separate step.
// Every barrier wait is bounded: a workgroup that waits longer than about a
// second raises the abort word and SPADE_DERR_SYNC, and every workgroup then
// leaves; the last one out resets the barrier words for the next launch.
#include "device_accept.h"
#include "device_attn.h"
#include "device_gemm.h"

namespace spade {

struct FusedParams {
  const uint8_t* weights;
  size_t layer_bytes, off_qkv, off_o, off_gu, off_down, off_g_attn, off_g_ffn, off_embed, off_g_final, off_lm;
  int L, d, H, F, V, Vpad;
  float eps, scale;
  uint8_t* kc;
  uint8_t* vc;
  size_t kv_layer_bytes;  // bytes between layers of the K (or V) cache
  uint32_t kv_bytes;      // bytes of one layer's K (or V) cache
  int kv_stride;
  const int32_t* lens;
  const int32_t* pending;
  int nb, R, M;
  const int32_t* drafts;
  const uint8_t* mode;
  const float* q;
  const float* u;
  float inv_T;
  int have_q;
  int32_t* n_out;
  int32_t* corr_out;
  float* logits;
  float* x;
  uint8_t* arena;  // FusedArena
  FusedArena fa;
  float* part_o;
  float* part_ml;
  uint32_t* attn_cnt;
  int NC, Rmax;
  float* stats;
  const float* rope;
  uint32_t* bar;
  uint32_t* err;
};

constexpr int kFusedThreads = 512;
constexpr int kHd = kAttnHd;  // head_dim of this path
constexpr uint64_t kSyncTimeoutTicks = 100000000ull;  // ~1 s of the 100 MHz wall clock

// barrier words (64 words apart): group counters 0..7, exit counter, abort flag
constexpr int kBarGroup = 0, kBarExit = 8 * 64, kBarAbort = 9 * 64;

__device__ __forceinline__ uint32_t ld_rlx(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_rlx(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_rlx(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh_u16(uint16_t* p, uint16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
struct GridSync {
  uint32_t* w;
  uint32_t epoch;
  int bid, G;
};

// Arrive at the next barrier: every store of this workgroup has completed.
__device__ __forceinline__ void sync_arrive(GridSync& s) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  ++s.epoch;
  if (threadIdx.x == 0) (void)add_rlx(s.w + kBarGroup + (s.bid & 7) * 64, 1u);
}

// Wait for every workgroup's arrival: lanes 0..7 of wave 0 poll the group
// counters (group x has (G - x + 7) / 8 members), lane 8 the abort word.
// False if the launch is aborting.
__device__ __forceinline__ bool sync_wait(GridSync& s, uint32_t* err, int* flag) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int x = lane & 7;
    const uint32_t target = s.epoch * (uint32_t)((s.G - x + 7) >> 3);
    int ok = 1;
    const uint64_t t0 = wall_clock64();
    while (true) {
      const uint32_t v = lane < 8 ? ld_rlx(s.w + kBarGroup + x * 64) : target;
      const uint32_t ab = lane == 8 ? ld_rlx(s.w + kBarAbort) : 0u;
      if (__all(v >= target)) break;
      if (__any(ab != 0u)) {
        ok = 0;
        break;
      }
      if (wall_clock64() - t0 > kSyncTimeoutTicks) {
        if (lane == 0) {
          st_rlx(s.w + kBarAbort, 1u);
          flag_error(err, SPADE_DERR_SYNC);
        }
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (lane == 0) *flag = ok;
  }
  __syncthreads();
  return *flag != 0;
}

// Leave the launch; the last workgroup out resets the barrier words (and, if
// the launch aborted, the attention arrival counters).
__device__ __forceinline__ void sync_exit(GridSync& s, uint32_t* attn_cnt, int n_cnt) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t o = add_rlx(s.w + kBarExit, 1u);
    if (o == (uint32_t)s.G - 1u) {
      const bool aborted = ld_rlx(s.w + kBarAbort) != 0u;
      if (aborted)
        for (int i = 0; i < n_cnt; ++i) st_rlx(attn_cnt + i, 0u);
      for (int x = 0; x < 8; ++x) st_rlx(s.w + kBarGroup + x * 64, 0u);
      st_rlx(s.w + kBarAbort, 0u);
      st_rlx(s.w + kBarExit, 0u);
    }
  }
}

// ---------------------------------------------------------------------------
// Embedding (Sec. III-A): x_0 = E[token] and the operand x_0 * g_attn of the
// first QKV projection, with per-16-column sums of squares.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void fused_embed(const FusedParams& P, int bid, int G) {
  const int total = P.M * P.d;
  const uint16_t* E = (const uint16_t*)(P.weights + P.off_embed);
  const float* g = (const float*)(P.weights + P.off_g_attn);  // layer 0
  uint16_t* act = (uint16_t*)(P.arena + P.fa.e_act);
  float* ssq = (float*)(P.arena + P.fa.e_ssq);
  const size_t split = (size_t)kFusedRows * P.d;
  // sixteen consecutive lanes hold the sixteen columns of one RMS partial
  for (int idx = bid * kFusedThreads + (int)threadIdx.x; idx < ((total + 63) & ~63); idx += G * kFusedThreads) {
    const bool ok = idx < total;
    const int m = ok ? idx / P.d : 0, n = ok ? idx - m * P.d : 0;
    const int bl = m / P.R, i = m - bl * P.R;
    int t = (i == 0) ? P.pending[bl] : P.drafts[bl * (P.R - 1) + i - 1];
    if (ok && (t < 0 || t >= P.V)) flag_error(P.err, SPADE_DERR_TOKEN);
    t = t < 0 ? 0 : (t >= P.V ? P.V - 1 : t);
    const float v = bf2f(E[(size_t)t * P.d + n]);
    float rem = v * g[n];
    float ss = v * v;
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    if (ok) {
      st_coh(P.x + (size_t)m * P.d + n, v);
#pragma unroll
      for (int s = 0; s < kActSplits; ++s) {
        const uint16_t h = f2bf(rem);
        st_coh_u16(act + s * split + (size_t)m * P.d + n, h);
        rem -= bf2f(h);
      }
      if ((n & 15) == 0) st_coh(ssq + (size_t)m * (P.d >> 4) + (n >> 4), ss);
    }
  }
}

// ---------------------------------------------------------------------------
// Projection GEMM stages.
// ---------------------------------------------------------------------------
template <int KIND>
__device__ __forceinline__ GemmParams fused_gemm_params(const FusedParams& P, int layer) {
  GemmParams g{};
  g.R = P.R;
  g.b0 = 0;
  g.lens = P.lens;
  g.inv_din = 1.0f / (float)P.d;
  g.eps = P.eps;
  g.n_ssq = P.d >> 4;
  g.H = P.H;
  g.Hkv = P.H;
  g.hd = kHd;
  g.d = P.d;
  g.F = P.F;
  g.kv_stride = P.kv_stride;
  g.kv_bf16 = 1;
  g.kv_bytes = P.kv_bytes;
  g.rope = P.rope;
  g.x = P.x;
  g.V = P.V;
  g.err = P.err;
  g.M = P.M;
  g.m0 = 0;
  const uint8_t* lb = P.weights + (size_t)layer * P.layer_bytes;
  uint8_t* ar = P.arena + (size_t)layer * P.fa.layer_bytes;          // this layer's block
  uint8_t* pr = layer > 0 ? ar - P.fa.layer_bytes : nullptr;       // the previous layer's
  const size_t sd = (size_t)kFusedRows * P.d, sf = (size_t)kFusedRows * P.F;
  int K;
  if constexpr (KIND == GEMM_QKV) {
    g.w = lb + P.off_qkv; K = P.d; g.n_units = 3 * P.d / 16; g.act_split = sd;
    g.act = layer > 0 ? (const void*)(pr + P.fa.act_nd) : (const void*)(P.arena + P.fa.e_act);
    g.ssq_in = layer > 0 ? (const float*)(pr + P.fa.ssq_d) : (const float*)(P.arena + P.fa.e_ssq);
    g.q_out = (float*)(ar + P.fa.q);
    g.kc = P.kc + (size_t)layer * P.kv_layer_bytes;
    g.vc = P.vc + (size_t)layer * P.kv_layer_bytes;
  } else if constexpr (KIND == GEMM_O) {
    g.w = lb + P.off_o; K = P.d; g.n_units = P.d / 16; g.act = ar + P.fa.act_o; g.act_split = sd;
    g.act_out = ar + P.fa.act_no;
    g.act_out_split = sd;
    g.act_out_stride = P.d;
    g.g_next = (const float*)(lb + P.off_g_ffn);
    g.ssq_out = (float*)(ar + P.fa.ssq_o);
    g.n_ssq_out = P.d >> 4;
  } else if constexpr (KIND == GEMM_GU) {
    g.w = lb + P.off_gu; K = P.d; g.n_units = 2 * P.F / 16; g.act = ar + P.fa.act_no; g.act_split = sd;
    g.ssq_in = (const float*)(ar + P.fa.ssq_o);
    g.act_out = ar + P.fa.act_f;
    g.act_out_split = sf;
    g.act_out_stride = P.F;
  } else if constexpr (KIND == GEMM_DOWN) {
    g.w = lb + P.off_down; K = P.F; g.n_units = P.d / 16; g.act = ar + P.fa.act_f; g.act_split = sf;
    g.act_out = ar + P.fa.act_nd;
    g.act_out_split = sd;
    g.act_out_stride = P.d;
    g.g_next = (layer + 1 < P.L) ? (const float*)(P.weights + (size_t)(layer + 1) * P.layer_bytes + P.off_g_attn)
                                 : (const float*)(P.weights + P.off_g_final);
    g.ssq_out = (float*)(ar + P.fa.ssq_d);
    g.n_ssq_out = P.d >> 4;
  } else {  // LM head on the last layer's output (called with layer = L - 1)
    g.w = P.weights + P.off_lm; K = P.d; g.n_units = P.Vpad / 16; g.act = ar + P.fa.act_nd; g.act_split = sd;
    g.ssq_in = (const float*)(ar + P.fa.ssq_d);
    g.logits = P.logits;
    g.stats = P.stats;
    g.NU = gridDim.x;  // one statistics entry per workgroup and row
    g.mode = P.mode;
    g.inv_T = P.inv_T;
    g.have_q = P.have_q;
  }
  g.NKB = K / 256;
  g.act_stride = K;
  return g;
}

// arrive (ending the previous stage), request the first weight tiles, wait, run
template <int KIND, bool ALDS>
__device__ __forceinline__ bool fused_gemm(const FusedParams& P, int layer, GridSync& gs, uint8_t* lds, int* flag) {
  const GemmParams gp = fused_gemm_params<KIND>(P, layer);
  Gemm<true, 1, ALDS, KIND, true> g(gp, *(GemmSmem<1>*)lds, lds + sizeof(GemmSmem<1>), gs.bid, gs.G);
  sync_arrive(gs);
  g.prefetch();
  if (!sync_wait(gs, P.err, flag)) return false;
  g.run();
  return true;
}

// ---------------------------------------------------------------------------
// Attention (device_attn.h): one (request, head, chunk) item per workgroup
// and round.  The cached keys older than this call are requested before the
// barrier that ends the QKV stage; the keys this call appended are read after
// it with sc1 loads.  Each chunk writes its partial (sc1), then arrives on the
// counter of its (request, head); the last arrival merges the chunks.
// ---------------------------------------------------------------------------
template <int CK>
struct FusedAttnSmem {
  AttnSmem<CK> a;
  AttnMergeSmem ms;
};

template <int CK>
__device__ __forceinline__ AttnItem fused_attn_item(const FusedParams& P, int layer, int item) {
  const int total = P.nb * P.H * P.NC;
  const bool valid = item < total;
  const int x = valid ? item : 0;
  const int c = x % P.NC, bh = x / P.NC;
  const int h = bh % P.H, bl = bh / P.H;
  return attn_item<CK>(valid, bl, h, c, P.lens[bl], P.R, P.kc + (size_t)layer * P.kv_layer_bytes,
                       P.vc + (size_t)layer * P.kv_layer_bytes, ((size_t)bl * P.H + h) * P.kv_stride * kAttnHd);
}

// keys older than this call: plain loads (may run before the barrier)
template <int CK>
__device__ __forceinline__ void fused_attn_prefetch(const FusedParams& P, const AttnItem& it, int wave, int lane,
                                                    AttnRegs<CK>& r) {
  attn_zero_regs(r);
  if (it.active) attn_load_plain(it, P.kv_stride, it.k_lo, min(it.k_hi, it.L), wave, lane, r);
}

template <int CK>
__device__ __forceinline__ void fused_attn_run(const FusedParams& P, int layer, const AttnItem& it, AttnRegs<CK>& r,
                                               FusedAttnSmem<CK>& sm, int wave, int lane) {
  const int R = P.R;
  const float* q = (const float*)(P.arena + (size_t)layer * P.fa.layer_bytes + P.fa.q) +
                   (size_t)(it.bl * R) * P.d + it.h * kAttnHd;
  float4 qr[8];
  attn_load_q(it, q, P.d, R, lane, qr);
  if (it.active) attn_load_new(it, wave_rsrc(it.kc), wave_rsrc(it.vc), P.kv_stride, wave, lane, r);
  attn_mask_tail(it, lane, r);
  const floatx4 o = attn_chunk(it, qr, R, P.scale, r, sm.a);
  // publish, arrive, and merge in the last arrival into this layer's O operand
  uint16_t* act = (uint16_t*)(P.arena + (size_t)layer * P.fa.layer_bytes + P.fa.act_o);
  const size_t split = (size_t)kFusedRows * P.d;
  attn_publish_merge(it, o, sm.a, sm.ms, P.part_o, P.part_ml, P.attn_cnt, P.H, P.NC, P.Rmax, R, [&](int oi, float O) {
    const int row = oi / kAttnHd, dd = oi - row * kAttnHd;
    const size_t e = (size_t)(it.bl * R + row) * P.d + it.h * kAttnHd + dd;
    float rem = O;
#pragma unroll
    for (int s = 0; s < kActSplits; ++s) {
      const uint16_t hb = f2bf(rem);
      st_coh_u16(act + s * split + e, hb);
      rem -= bf2f(hb);
    }
  });
}

template <int CK>
__device__ __forceinline__ bool fused_attention(const FusedParams& P, int layer, GridSync& gs, uint8_t* lds,
                                                int* flag) {
  FusedAttnSmem<CK>& sm = *(FusedAttnSmem<CK>*)lds;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
  const int total = P.nb * P.H * P.NC;
  const int rounds = (total + gs.G - 1) / gs.G;
  AttnRegs<CK> r;
  AttnItem it = fused_attn_item<CK>(P, layer, gs.bid);
  sync_arrive(gs);
  fused_attn_prefetch(P, it, wave, lane, r);
  if (!sync_wait(gs, P.err, flag)) return false;
  for (int k = 0; k < rounds; ++k) {
    if (k > 0) {
      it = fused_attn_item<CK>(P, layer, k * gs.G + gs.bid);
      fused_attn_prefetch(P, it, wave, lane, r);
    }
    fused_attn_run(P, layer, it, r, sm, wave, lane);
    __syncthreads();  // the next round reuses the LDS
  }
  return true;
}

// ---------------------------------------------------------------------------
// The kernel.
// ---------------------------------------------------------------------------
template <bool LDS_D, bool LDS_F, int CK>
__global__ void __launch_bounds__(kFusedThreads) verify_fused_kernel(FusedParams P) {
  extern __shared__ uint4 lds_raw[];
  uint8_t* lds = (uint8_t*)lds_raw;
  __shared__ int flag;
  GridSync gs{P.bar, 0u, (int)blockIdx.x, (int)gridDim.x};
  bool ok = true;

  fused_embed(P, gs.bid, gs.G);
  for (int l = 0; l < P.L && ok; ++l) {
    ok = fused_gemm<GEMM_QKV, LDS_D>(P, l, gs, lds, &flag);
    if (ok) ok = fused_attention<CK>(P, l, gs, lds, &flag);
    if (ok) ok = fused_gemm<GEMM_O, LDS_D>(P, l, gs, lds, &flag);
    if (ok) ok = fused_gemm<GEMM_GU, LDS_D>(P, l, gs, lds, &flag);
    if (ok) ok = fused_gemm<GEMM_DOWN, LDS_F>(P, l, gs, lds, &flag);
  }
  if (ok) ok = fused_gemm<GEMM_LM, LDS_D>(P, P.L - 1, gs, lds, &flag);
  if (ok) {
    sync_arrive(gs);
    ok = sync_wait(gs, P.err, &flag);
  }
  if (ok && gs.bid < P.nb) {
    AcceptParams ap{};
    ap.logits = P.logits;
    ap.stats = P.stats;
    ap.NU = gs.G;
    ap.V = P.V;
    ap.gamma = P.R - 1;
    ap.R = P.R;
    ap.drafts = P.drafts;
    ap.q = P.q;
    ap.u = P.u;
    ap.mode = P.mode;
    ap.inv_T = P.inv_T;
    ap.n_out = P.n_out;
    ap.corr_out = P.corr_out;
    ap.err = P.err;
    accept_request<kFusedThreads, false>(ap, gs.bid, *(AcceptSmem*)lds);
  }
  sync_exit(gs, P.attn_cnt, P.nb * P.H);
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
namespace {

template <bool LDS_D, bool LDS_F, int CK>
hipError_t launch_fused_t(const FusedParams& p, int grid, uint32_t lds, hipStream_t st) {
  const void* fn = reinterpret_cast<const void*>(&verify_fused_kernel<LDS_D, LDS_F, CK>);
  static hipError_t attr = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kFusedLdsBytes);
  if (attr != hipSuccess) return attr;
  FusedParams arg = p;
  void* args[] = {&arg};
  return hipLaunchCooperativeKernel(fn, dim3(grid), dim3(kFusedThreads), args, lds, st);
}

}  // namespace

bool fused_eligible(spade_model md, spade_kv kv, const ForwardCall& fc) {
  const Dims& D = md->dims;
  if (!md->fused_ok || md->ws.fused == nullptr) return false;
  if (D.wdt != SPADE_BF16 || D.kvdt != SPADE_BF16 || D.hd != kHd) return false;
  if (D.KVH != D.H) return false;  // multi-head attention only
  if (fc.tokens != nullptr || fc.b0 != 0 || !fc.want_logits) return false;
  const int M = fc.nb * fc.R;
  if (M > kFusedRows || fc.R > kAttnRows) return false;
  const size_t kv_layer = (size_t)kv->max_batch * D.H * kv->stride * D.hd * 2;
  if (kv_layer >= (1ull << 31)) return false;
  return true;
}

hipError_t launch_verify_fused(spade_model md, spade_kv kv, const ForwardCall& fc, const AcceptCall& ac,
                               hipStream_t st) {
  const Dims& D = md->dims;
  const Workspace& W = md->ws;
  int max_keys = 0;
  for (int b = 0; b < fc.nb; ++b) max_keys = std::max(max_keys, kv->lens_ub[b] + fc.R);
  constexpr int CK = kAttnChunkKeys;  // as the per-stage path
  const int NC = (max_keys + CK - 1) / CK;
  if (NC > W.NCmax || NC > kAttnMaxChunks) return hipErrorInvalidValue;

  FusedParams p{};
  p.weights = md->weights;
  p.layer_bytes = md->lay.layer_bytes;
  p.off_qkv = md->lay.qkv;
  p.off_o = md->lay.o;
  p.off_gu = md->lay.gu;
  p.off_down = md->lay.down;
  p.off_g_attn = md->lay.g_attn;
  p.off_g_ffn = md->lay.g_ffn;
  p.off_embed = md->lay.embed;
  p.off_g_final = md->lay.g_final;
  p.off_lm = md->lay.lm;
  p.L = D.L;
  p.d = D.d;
  p.H = D.H;
  p.F = D.F;
  p.V = D.V;
  p.Vpad = D.Vpad;
  p.eps = D.eps;
  p.scale = 1.0f / sqrtf((float)D.hd);
  p.kc = kv->k;
  p.vc = kv->v;
  p.kv_layer_bytes = (size_t)kv->max_batch * D.H * kv->stride * D.hd * 2;
  p.kv_bytes = (uint32_t)p.kv_layer_bytes;
  p.kv_stride = kv->stride;
  p.lens = kv->lens;
  p.pending = kv->pending;
  p.nb = fc.nb;
  p.R = fc.R;
  p.M = fc.nb * fc.R;
  p.drafts = fc.drafts;
  p.mode = fc.mode;
  p.q = ac.q;
  p.u = ac.u;
  p.inv_T = fc.inv_T;
  p.have_q = fc.have_q;
  p.n_out = ac.n_out;
  p.corr_out = ac.corr_out;
  p.logits = fc.logits_out;
  p.x = W.x;
  p.arena = W.fused;
  p.fa = W.fa;
  p.part_o = W.attn_o;
  p.part_ml = W.attn_ml;
  p.attn_cnt = W.attn_cnt;
  p.NC = NC;
  p.Rmax = W.Rmax;
  p.stats = W.stats;
  p.rope = W.rope;
  p.bar = W.bar;
  p.err = W.err;

  const uint32_t gsm = (uint32_t)sizeof(GemmSmem<1>);
  const uint32_t lds_d = gsm + gemm_lds_a_bytes(p.M, D.d, 1);
  const uint32_t lds_f = gsm + gemm_lds_a_bytes(p.M, D.F, 1);
  const bool use_d = lds_d <= kFusedLdsBytes && gemm_lds_a_ok(D.d, 1);
  const bool use_f = lds_f <= kFusedLdsBytes && gemm_lds_a_ok(D.F, 1);
  uint32_t lds = (uint32_t)std::max(sizeof(FusedAttnSmem<CK>), sizeof(AcceptSmem));
  lds = std::max(lds, gsm);
  if (use_d) lds = std::max(lds, lds_d);
  if (use_f) lds = std::max(lds, lds_f);
  lds = (lds + 15) / 16 * 16;
  const int grid = md->n_cu;
  if (use_d && use_f) return launch_fused_t<true, true, CK>(p, grid, lds, st);
  if (use_d) return launch_fused_t<true, false, CK>(p, grid, lds, st);
  if (use_f) return launch_fused_t<false, true, CK>(p, grid, lds, st);
  return launch_fused_t<false, false, CK>(p, grid, lds, st);
}

}  // namespace spade
