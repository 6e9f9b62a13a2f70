// C ABI of the speculative-verify library: argument checks, memory layout of
// the caller's buffers, and the launch sequence of one call.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "spade_internal.h"

using namespace spade;

namespace {

thread_local char g_err[512] = "";

spade_status fail(spade_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

spade_status hipfail(hipError_t e, const char* what) {
  return fail(SPADE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Set the host bound of lens[0..B) to the device values (synchronises).
spade_status refresh_bound(spade_kv kv, int B, hipStream_t st) {
  std::vector<int32_t> h(B);
  hipError_t e = hipMemcpyAsync(h.data(), kv->lens, (size_t)B * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hipfail(e, "reading lens");
  for (int b = 0; b < B; ++b) kv->lens_ub[b] = std::max(0, (int)h[b]);
  return SPADE_OK;
}

spade_status check_config(const spade_config* c) {
  if (!c) return fail(SPADE_EINVAL, "null config");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->head_dim < 1 || c->d_ffn < 1 || c->vocab < 2)
    return fail(SPADE_EINVAL, "config dimensions must be positive (vocab >= 2)");
  if (c->weight_dtype != SPADE_BF16 && c->weight_dtype != SPADE_F32)
    return fail(SPADE_EINVAL, "weight_dtype must be SPADE_BF16 or SPADE_F32");
  if (c->kv_dtype != SPADE_BF16 && c->kv_dtype != SPADE_F32)
    return fail(SPADE_EINVAL, "kv_dtype must be SPADE_BF16 or SPADE_F32");
  if (c->d_model != c->n_heads * c->head_dim) return fail(SPADE_EINVAL, "d_model != n_heads * head_dim");
  if (c->n_kv_heads < 0 || (c->n_kv_heads > 0 && c->n_heads % c->n_kv_heads != 0))
    return fail(SPADE_EINVAL, "n_kv_heads must be 0 or a divisor of n_heads");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(SPADE_EUNSUPPORTED, "head_dim must be 64 or 128");
  const int kb = kblock_of(c->weight_dtype);
  if (c->d_model % kb || c->d_ffn % kb)
    return fail(SPADE_EUNSUPPORTED, "d_model and d_ffn must be multiples of %d for this weight dtype", kb);
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail(SPADE_EINVAL, "bad rms_eps / rope_theta");
  return SPADE_OK;
}

Dims dims_of(const spade_config* c) {
  Dims d{};
  d.L = c->n_layers;
  d.d = c->d_model;
  d.H = c->n_heads;
  d.hd = c->head_dim;
  d.KVH = c->n_kv_heads > 0 ? c->n_kv_heads : c->n_heads;
  d.dkv = d.KVH * c->head_dim;
  d.F = c->d_ffn;
  d.V = c->vocab;
  d.Vpad = (c->vocab + 15) / 16 * 16;
  d.wdt = c->weight_dtype;
  d.kvdt = c->kv_dtype;
  d.eps = c->rms_eps;
  d.theta = c->rope_theta;
  return d;
}

ArenaLayout layout_of(const Dims& D) {
  const size_t e = D.wdt == SPADE_BF16 ? 2 : 4;
  ArenaLayout a{};
  size_t off = 0;
  a.qkv = off;  off += align256((size_t)(D.d + 2 * D.dkv) * D.d * e);
  a.o = off;    off += align256((size_t)D.d * D.d * e);
  a.gu = off;   off += align256((size_t)2 * D.F * D.d * e);
  a.down = off; off += align256((size_t)D.d * D.F * e);
  a.g_attn = off; off += align256((size_t)D.d * 4);
  a.g_ffn = off;  off += align256((size_t)D.d * 4);
  a.layer_bytes = off;
  off = a.layer_bytes * D.L;
  a.embed = off;   off += align256((size_t)D.V * D.d * e);
  a.g_final = off; off += align256((size_t)D.d * 4);
  a.lm = off;      off += align256((size_t)D.Vpad * D.d * e);
  a.total = off;
  return a;
}

struct WsPlan {
  size_t x, act_n, act_o, act_f, ssq, q, attn_o, attn_ml, attn_cnt, logits, stats, rope, err, split_cnt,
      split_part, wide_cnt, wide_part, mid_part, corr_lse, corr_part, corr_cnt, prefill_tok, prefill_cnt, prefill_base, total;
  size_t wide_items, wide_floats, mid_items;
  int max_units;
  size_t act_split, actf_split;
  int Mmax, Mrows, NCmax, Rmax;
};

WsPlan plan_ws(const Dims& D, int max_batch, int max_gamma, int max_len) {
  WsPlan p{};
  p.Rmax = std::max(max_gamma + 1, kPrefillRows);
  // rows of a verify call, or of a batched prefill of 16 tokens per request
  p.Mmax = std::max(max_batch * (max_gamma + 1), max_batch * kPrefillRows);
  // rows of any forward: a bf16 cache with head_dim 128 also takes prefill
  // forwards of up to kPrefillMaxRows prompt rows (no more than the caches hold)
  p.Mrows = p.Mmax;
  if (D.kvdt == SPADE_BF16 && D.hd == kAttnHd)
    p.Mrows = std::max(p.Mmax, (int)std::min<long>(kPrefillMaxRows, (long)max_batch * ((max_len + 15) / 16 * 16)));
  p.NCmax = std::min(kAttnMaxChunks, (max_len + kAttnChunk - 1) / kAttnChunk);
  const bool wb = D.wdt == SPADE_BF16;
  const size_t ae = wb ? 2 * kActSplits : 4;  // bf16 terms or one float
  p.act_split = (size_t)p.Mrows * D.d;
  p.actf_split = (size_t)p.Mrows * D.F;
  const int NU = D.Vpad / 16;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  p.x = take((size_t)p.Mrows * D.d * 4);
  p.act_n = take((size_t)p.Mrows * D.d * ae);
  p.act_o = take((size_t)p.Mrows * D.d * ae);
  p.act_f = take((size_t)p.Mrows * D.F * ae);
  p.ssq = take((size_t)p.Mrows * (D.d / 16) * 4);
  p.q = take((size_t)p.Mrows * D.d * 4);
  p.attn_o = take((size_t)max_batch * D.H * p.NCmax * p.Rmax * D.hd * 4);
  p.attn_ml = take((size_t)max_batch * D.H * p.NCmax * p.Rmax * 2 * 4);
  p.attn_cnt = take((size_t)max_batch * D.H * 4);
  p.logits = take((size_t)p.Mmax * D.V * 4);
  p.stats = take((size_t)p.Mmax * std::max(NU, kMaxStatGroups) * 3 * 4);  // NU = panels of the LM head
  p.rope = take((size_t)max_len * (D.hd / 2) * 2 * 4);
  p.err = take(4);
  p.max_units = std::max(std::max(D.d + 2 * D.dkv, 2 * D.F), D.Vpad) / 16;
  p.split_cnt = take((size_t)p.max_units * 4);
  p.split_part = take((size_t)p.max_units * 8 * 256 * 4);
  // k-split wide-row O and down projections (d / 16 panels, up to Mmax rows):
  // the most (unit group, row group) items and published floats any tiling needs
  if (wb) {
    const int nu = D.d / 16;
    // unit groups of 8 panels (one per wave) x row groups of one 16-row tile
    p.wide_items = (size_t)((nu + 7) / 8) * (size_t)((p.Mmax + 15) / 16);
    for (int rt = 1; rt <= 3; ++rt)
      for (int pp = 1; pp <= 2; ++pp)
        if (!(pp == 2 && rt == 3)) p.wide_floats = std::max(p.wide_floats, wide_split_floats(nu, p.Mmax, rt, pp));
  }
  p.wide_cnt = take(p.wide_items * 4);
  p.wide_part = take(p.wide_floats * 4);
  // medium-M projections (forwards of 17 to 144 rows): one block of published
  // sums per 256-column panel group of the widest projection
  if (wb && p.Mrows > kWideMinRows)
    p.mid_items = (size_t)((std::max(D.d + 2 * D.dkv, 2 * D.F) / 16 + 15) / 16);
  p.mid_part = take(p.mid_items * mid_split_floats() * 4);
  p.corr_lse = take((size_t)max_batch * 4);
  p.corr_part = take((size_t)max_batch * kCorrMaxSlices * 4 * 4);
  p.corr_cnt = take((size_t)max_batch * 4);
  p.prefill_tok = take((size_t)p.Mrows * 4);
  p.prefill_cnt = take((size_t)max_batch * 4);
  p.prefill_base = take((size_t)max_batch * 4);
  p.total = off;
  return p;
}

}  // namespace

extern "C" {

const char* spade_last_error(void) { return g_err; }

size_t spade_weight_bytes(const spade_config* cfg) {
  if (check_config(cfg) != SPADE_OK) return 0;
  return layout_of(dims_of(cfg)).total;
}

size_t spade_workspace_bytes(const spade_config* cfg, int max_batch, int max_gamma, int max_len) {
  if (check_config(cfg) != SPADE_OK || max_batch < 1 || max_gamma < 0 || max_gamma + 1 > kMaxR || max_len < 1)
    return 0;
  return plan_ws(dims_of(cfg), max_batch, max_gamma, max_len).total;
}

size_t spade_kv_bytes(const spade_config* cfg, int max_batch, int max_len) {
  if (check_config(cfg) != SPADE_OK || max_batch < 1 || max_len < 1) return 0;
  const size_t e = cfg->kv_dtype == SPADE_BF16 ? 2 : 4;
  const int kvh = cfg->n_kv_heads > 0 ? cfg->n_kv_heads : cfg->n_heads;
  return 2 * align256((size_t)cfg->n_layers * max_batch * kvh * kv_stride_of(max_len) * cfg->head_dim * e);
}

spade_status spade_model_create(const spade_config* cfg, void* d_weights, void* d_workspace, int max_batch,
                                int max_gamma, int max_len, spade_model* out) {
  spade_status s = check_config(cfg);
  if (s != SPADE_OK) return s;
  if (!d_weights || !d_workspace || !out) return fail(SPADE_EINVAL, "null pointer");
  if (((uintptr_t)d_weights | (uintptr_t)d_workspace) & 255) return fail(SPADE_EINVAL, "buffers must be 256-byte aligned");
  if (max_batch < 1 || max_len < 2) return fail(SPADE_EINVAL, "max_batch >= 1 and max_len >= 2 required");
  if (max_len > kMaxLen) return fail(SPADE_ECAPACITY, "max_len must be <= %d", kMaxLen);
  if (max_gamma < 0 || max_gamma + 1 > kMaxR) return fail(SPADE_ECAPACITY, "max_gamma must be in [0, %d]", kMaxR - 1);
  spade_model m = new (std::nothrow) spade_model_s();
  if (!m) return fail(SPADE_EINVAL, "out of host memory");
  m->cfg = *cfg;
  m->dims = dims_of(cfg);
  m->lay = layout_of(m->dims);
  m->weights = (uint8_t*)d_weights;
  m->work = (uint8_t*)d_workspace;
  m->max_batch = max_batch;
  m->max_gamma = max_gamma;
  m->max_len = max_len;
  (void)hipGetDevice(&m->device);
  m->n_cu = 0;
  if (hipDeviceGetAttribute(&m->n_cu, hipDeviceAttributeMultiprocessorCount, m->device) != hipSuccess ||
      m->n_cu < 1)
    m->n_cu = 256;
  // one 8-wave GEMM workgroup per compute unit (the kernel needs two waves per
  // SIMD); SPADE_GEMM_WGS overrides for experiments
  m->gemm_wgs = m->n_cu;
  m->wide_rt = 0;
  m->wide_p = 0;
  m->wide_ks = 0;
  m->split_ks = 0;
  m->attn_merge = 0;
  m->corr_split = 0;
  m->attn_grouped = 0;
  m->prefill_rows = 0;
  m->big_gemm = 0;
  m->mid_gemm = 0;
  m->mid_ks = 0;
  if (const char* ev = std::getenv("SPADE_GEMM_WGS")) {
    const int v = std::atoi(ev);
    if (v > 0) m->gemm_wgs = std::min(v, kMaxStatGroups);
  }
  const WsPlan p = plan_ws(m->dims, max_batch, max_gamma, max_len);
  Workspace& w = m->ws;
  uint8_t* b = m->work;
  w.x = (float*)(b + p.x);
  w.act_n = b + p.act_n;
  w.act_o = b + p.act_o;
  w.act_f = b + p.act_f;
  w.ssq = (float*)(b + p.ssq);
  w.q = (float*)(b + p.q);
  w.attn_o = (float*)(b + p.attn_o);
  w.attn_ml = (float*)(b + p.attn_ml);
  w.attn_cnt = (uint32_t*)(b + p.attn_cnt);
  w.split_cnt = (uint32_t*)(b + p.split_cnt);
  w.split_part = (float*)(b + p.split_part);
  w.wide_cnt = (uint32_t*)(b + p.wide_cnt);
  w.wide_part = (float*)(b + p.wide_part);
  w.wide_items = p.wide_items;
  w.wide_floats = p.wide_floats;
  w.mid_items = p.mid_items;
  w.mid_part = p.mid_items > 0 ? (float*)(b + p.mid_part) : nullptr;
  w.corr_lse = (float*)(b + p.corr_lse);
  w.corr_part = (float*)(b + p.corr_part);
  w.corr_cnt = (uint32_t*)(b + p.corr_cnt);
  w.prefill_tok = (int32_t*)(b + p.prefill_tok);
  w.prefill_cnt = (int32_t*)(b + p.prefill_cnt);
  w.prefill_base = (int32_t*)(b + p.prefill_base);
  w.logits = (float*)(b + p.logits);
  w.stats = (float*)(b + p.stats);
  w.rope = (float*)(b + p.rope);
  w.err = (uint32_t*)(b + p.err);
  w.act_split = p.act_split;
  w.actf_split = p.actf_split;
  w.Mmax = p.Mmax;
  w.Mrows = p.Mrows;
  w.NCmax = p.NCmax;
  w.Rmax = p.Rmax;

  // RoPE table: angle pos * theta^(-2i/hd) in double, stored as float.
  const int half = m->dims.hd / 2;
  std::vector<float> rope((size_t)max_len * half * 2);
  for (int pos = 0; pos < max_len; ++pos)
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow((double)cfg->rope_theta, -2.0 * i / (double)m->dims.hd);
      const double ang = (double)pos * inv;
      rope[((size_t)pos * half + i) * 2] = (float)std::cos(ang);
      rope[((size_t)pos * half + i) * 2 + 1] = (float)std::sin(ang);
    }
  hipError_t e = hipMemcpy(w.rope, rope.data(), rope.size() * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemset(w.attn_cnt, 0, (size_t)max_batch * m->dims.H * 4);
  if (e == hipSuccess) e = hipMemset(w.split_cnt, 0, (size_t)p.max_units * 4);
  if (e == hipSuccess && p.wide_items > 0) e = hipMemset(w.wide_cnt, 0, p.wide_items * 4);
  if (e == hipSuccess) e = hipMemset(w.corr_cnt, 0, (size_t)max_batch * 4);
  if (e == hipSuccess) e = hipMemset(w.err, 0, 4);
  // activation buffers start at zero so rows past M never feed NaNs
  if (e == hipSuccess) e = hipMemset(b, 0, p.ssq);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    delete m;
    return hipfail(e, "model_create");
  }
  *out = m;
  return SPADE_OK;
}

void spade_model_destroy(spade_model m) { delete m; }

spade_status spade_model_load_tensor(spade_model m, int kind, int layer, const void* d_src, void* stream) {
  if (!m || !d_src) return fail(SPADE_EINVAL, "null pointer");
  if (kind < SPADE_WQ || kind > SPADE_LM_HEAD) return fail(SPADE_EINVAL, "bad tensor kind %d", kind);
  const bool global = kind == SPADE_EMBED || kind == SPADE_G_FINAL || kind == SPADE_LM_HEAD;
  if (!global && (layer < 0 || layer >= m->dims.L)) return fail(SPADE_EINVAL, "layer %d out of range", layer);
  hipError_t e = launch_pack(m, kind, global ? 0 : layer, d_src, (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "load_tensor");
  return SPADE_OK;
}

spade_status spade_kv_create(spade_model m, void* d_kv, int max_batch, int max_len, int32_t* d_lens,
                             int32_t* d_pending, spade_kv* out) {
  if (!m || !d_kv || !d_lens || !d_pending || !out) return fail(SPADE_EINVAL, "null pointer");
  if ((uintptr_t)d_kv & 255) return fail(SPADE_EINVAL, "KV buffer must be 256-byte aligned");
  if (max_batch < 1 || max_batch > m->max_batch) return fail(SPADE_ECAPACITY, "kv max_batch exceeds the model's");
  if (max_len < 2 || max_len > m->max_len) return fail(SPADE_ECAPACITY, "kv max_len exceeds the model's");
  spade_kv kv = new (std::nothrow) spade_kv_s();
  if (!kv) return fail(SPADE_EINVAL, "out of host memory");
  kv->model = m;
  const size_t half = spade_kv_bytes(&m->cfg, max_batch, max_len) / 2;
  kv->k = (uint8_t*)d_kv;
  kv->v = (uint8_t*)d_kv + half;
  kv->lens = d_lens;
  kv->pending = d_pending;
  kv->max_batch = max_batch;
  kv->max_len = max_len;
  kv->stride = kv_stride_of(max_len);
  kv->lens_ub = new (std::nothrow) int[max_batch]();
  kv->last_rows = m->max_gamma + 1;
  kv->last_B = 0;
  kv->verified = false;
  kv->snap_ub = new (std::nothrow) int[max_batch]();
  if (!kv->lens_ub || !kv->snap_ub) {
    delete[] kv->lens_ub;
    delete[] kv->snap_ub;
    delete kv;
    return fail(SPADE_EINVAL, "out of host memory");
  }
  *out = kv;
  return SPADE_OK;
}

void spade_kv_destroy(spade_kv kv) {
  if (!kv) return;
  delete[] kv->lens_ub;
  delete[] kv->snap_ub;
  delete kv;
}

spade_status spade_kv_set_state(spade_kv kv, int B, const int32_t* h_lens, const int32_t* h_pending, void* stream) {
  if (!kv || !h_lens || !h_pending) return fail(SPADE_EINVAL, "null pointer");
  if (B < 1 || B > kv->max_batch) return fail(SPADE_ECAPACITY, "B out of range");
  for (int b = 0; b < B; ++b) {
    if (h_lens[b] < 0 || h_lens[b] >= kv->max_len) return fail(SPADE_ECAPACITY, "lens[%d] out of range", b);
    if (h_pending[b] < 0 || h_pending[b] >= kv->model->dims.V) return fail(SPADE_EINVAL, "pending[%d] out of range", b);
  }
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(kv->lens, h_lens, (size_t)B * 4, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipMemcpyAsync(kv->pending, h_pending, (size_t)B * 4, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hipfail(e, "kv_set_state");
  for (int b = 0; b < B; ++b) kv->lens_ub[b] = h_lens[b];
  kv->verified = false;
  return SPADE_OK;
}

spade_status spade_kv_get_state(spade_kv kv, int B, int32_t* h_lens, int32_t* h_pending, void* stream) {
  if (!kv || !h_lens || !h_pending) return fail(SPADE_EINVAL, "null pointer");
  if (B < 1 || B > kv->max_batch) return fail(SPADE_ECAPACITY, "B out of range");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(h_lens, kv->lens, (size_t)B * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipMemcpyAsync(h_pending, kv->pending, (size_t)B * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hipfail(e, "kv_get_state");
  for (int b = 0; b < B; ++b) kv->lens_ub[b] = h_lens[b];
  return SPADE_OK;
}

spade_status spade_kv_snapshot(spade_kv kv, int B, int32_t* d_lens, int32_t* d_pending, void* stream) {
  if (!kv || !d_lens || !d_pending) return fail(SPADE_EINVAL, "null pointer");
  if (B < 1 || B > kv->max_batch) return fail(SPADE_ECAPACITY, "B out of range");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = launch_copy_state(B, d_lens, d_pending, kv->lens, kv->pending, st);
  if (e != hipSuccess) return hipfail(e, "kv_snapshot");
  for (int b = 0; b < kv->max_batch; ++b) kv->snap_ub[b] = kv->lens_ub[b];
  return SPADE_OK;
}

spade_status spade_kv_restore(spade_kv kv, int B, const int32_t* d_lens, const int32_t* d_pending, void* stream) {
  if (!kv || !d_lens || !d_pending) return fail(SPADE_EINVAL, "null pointer");
  if (B < 1 || B > kv->max_batch) return fail(SPADE_ECAPACITY, "B out of range");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = launch_copy_state(B, kv->lens, kv->pending, d_lens, d_pending, st);
  if (e != hipSuccess) return hipfail(e, "kv_restore");
  for (int b = 0; b < B; ++b) kv->lens_ub[b] = kv->snap_ub[b];
  kv->verified = false;
  return SPADE_OK;
}

spade_status spade_prefill(spade_model m, spade_kv kv, int b, const int32_t* d_tokens, int n_tokens, void* stream) {
  if (!m || !kv || !d_tokens) return fail(SPADE_EINVAL, "null pointer");
  if (kv->model != m) return fail(SPADE_EINVAL, "kv belongs to another model");
  if (b < 0 || b >= kv->max_batch) return fail(SPADE_EINVAL, "request %d out of range", b);
  if (n_tokens < 1) return fail(SPADE_EINVAL, "n_tokens must be >= 1");
  const int n_cache = n_tokens - 1;
  if (kv->lens_ub[b] + n_cache + 1 > kv->max_len)
    return fail(SPADE_ECAPACITY, "prefill of %d tokens overflows max_len %d", n_tokens, kv->max_len);
  hipError_t e = launch_prefill_one(m, kv, b, d_tokens, n_cache, (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "prefill");
  kv->verified = false;
  return SPADE_OK;
}

spade_status spade_verify(spade_model m, spade_kv kv, int B, int gamma, const int32_t* d_draft_tokens,
                          const float* d_draft_probs, const float* d_uniforms, const uint8_t* d_mode,
                          float temperature, int32_t* d_n_accepted, int32_t* d_correction, float* d_logits,
                          void* stream) {
  if (!m || !kv || !d_mode || !d_n_accepted || !d_correction) return fail(SPADE_EINVAL, "null pointer");
  if (kv->model != m) return fail(SPADE_EINVAL, "kv belongs to another model");
  if (B < 1 || B > m->max_batch || B > kv->max_batch) return fail(SPADE_ECAPACITY, "B=%d out of range", B);
  if (gamma < 0 || gamma > m->max_gamma) return fail(SPADE_ECAPACITY, "gamma=%d out of range", gamma);
  if (gamma > 0 && !d_draft_tokens) return fail(SPADE_EINVAL, "draft tokens required when gamma > 0");
  if (d_draft_probs && !d_uniforms) return fail(SPADE_EINVAL, "sampling needs uniforms");
  if (!(temperature > 0.f && std::isfinite(temperature)))
    return fail(SPADE_EINVAL, "temperature must be finite and > 0");
  hipStream_t st = (hipStream_t)stream;
  bool refreshed = false;
  for (int b = 0; b < B; ++b)
    if (kv->lens_ub[b] + gamma + 1 > kv->max_len) {
      // the host bound grows by gamma + 1 per commit while the lengths grow
      // by k + 1: read the device lengths once before giving up
      if (!refreshed) {
        spade_status rs = refresh_bound(kv, B, st);
        if (rs != SPADE_OK) return rs;
        refreshed = true;
      }
      if (kv->lens_ub[b] + gamma + 1 > kv->max_len)
        return fail(SPADE_ECAPACITY, "request %d: %d cached + %d rows exceed max_len %d", b, kv->lens_ub[b],
                    gamma + 1, kv->max_len);
    }
  kv->last_rows = gamma + 1;
  kv->last_B = B;
  kv->verified = true;
  ForwardCall fc{};
  fc.b0 = 0;
  fc.nb = B;
  fc.R = gamma + 1;
  fc.drafts = d_draft_tokens;
  fc.want_logits = true;
  fc.logits_out = d_logits ? d_logits : m->ws.logits;
  fc.mode = d_mode;
  fc.inv_T = 1.0f / temperature;
  fc.have_q = d_uniforms != nullptr && (d_draft_probs != nullptr || gamma == 0);
  AcceptCall ac{};
  ac.B = B;
  ac.gamma = gamma;
  ac.V = m->dims.V;
  ac.logits = fc.logits_out;
  ac.stats = m->ws.stats;
  ac.NU = std::min(m->dims.Vpad / 16, m->gemm_wgs);  // LM-head workgroups
  ac.panels = lm_stats_panels(m, B * (gamma + 1));
  ac.drafts = d_draft_tokens;
  ac.q = d_draft_probs;
  ac.u = d_uniforms;
  ac.mode = d_mode;
  ac.inv_T = fc.inv_T;
  ac.n_out = d_n_accepted;
  ac.corr_out = d_correction;
  hipError_t e = launch_forward(m, kv, fc, st);
  if (e == hipSuccess) e = launch_accept(m, ac, st);
  if (e != hipSuccess) return hipfail(e, "verify");
  return SPADE_OK;
}

spade_status spade_model_set_wide_tiles(spade_model m, int row_tiles, int panels) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (row_tiles < -1 || row_tiles > 3) return fail(SPADE_EINVAL, "row_tiles must be -1, 0, 1, 2 or 3");
  if (panels < 0 || panels > 2) return fail(SPADE_EINVAL, "panels must be 0, 1 or 2");
  m->wide_rt = row_tiles;
  m->wide_p = panels;
  return SPADE_OK;
}

spade_status spade_model_set_attn_merge(spade_model m, int mode) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (mode < 0 || mode > 2) return fail(SPADE_EINVAL, "mode must be 0, 1 or 2");
  m->attn_merge = mode;
  return SPADE_OK;
}

spade_status spade_model_set_attn_grouped(spade_model m, int mode) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (mode < 0 || mode > 1) return fail(SPADE_EINVAL, "mode must be 0 or 1");
  m->attn_grouped = mode;
  return SPADE_OK;
}

spade_status spade_model_set_prefill_rows(spade_model m, int rows) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (rows < 0) return fail(SPADE_EINVAL, "rows must be >= 0");
  m->prefill_rows = rows;
  return SPADE_OK;
}

spade_status spade_model_set_big_gemm(spade_model m, int mode) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (mode < 0 || mode > 2) return fail(SPADE_EINVAL, "mode must be 0, 1 or 2");
  m->big_gemm = mode;
  return SPADE_OK;
}

spade_status spade_model_set_mid_gemm(spade_model m, int mode, int k_splits) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (mode < 0 || mode > 2) return fail(SPADE_EINVAL, "mode must be 0, 1 or 2");
  if (k_splits < 0 || k_splits > 8) return fail(SPADE_EINVAL, "k_splits must be 0..8");
  m->mid_gemm = mode;
  m->mid_ks = k_splits;
  return SPADE_OK;
}

spade_status spade_model_set_correction_slices(spade_model m, int mode) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (mode < 0 || mode > 2) return fail(SPADE_EINVAL, "mode must be 0, 1 or 2");
  m->corr_split = mode;
  return SPADE_OK;
}

spade_status spade_model_set_wide_k_splits(spade_model m, int splits) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (splits != 0 && splits != 1 && splits != 2 && splits != 4) return fail(SPADE_EINVAL, "splits must be 0, 1, 2 or 4");
  m->wide_ks = splits;
  return SPADE_OK;
}

spade_status spade_prefill_batch(spade_model m, spade_kv kv, int B, const int32_t* d_tokens, int ld,
                                 const int32_t* h_n_tokens, void* stream) {
  if (!m || !kv || !d_tokens || !h_n_tokens) return fail(SPADE_EINVAL, "null pointer");
  if (kv->model != m) return fail(SPADE_EINVAL, "kv belongs to another model");
  if (B < 1 || B > kv->max_batch || B > m->max_batch) return fail(SPADE_ECAPACITY, "B=%d out of range", B);
  std::vector<int> n_cache(B);
  for (int b = 0; b < B; ++b) {
    if (h_n_tokens[b] < 1 || h_n_tokens[b] > ld) return fail(SPADE_EINVAL, "request %d: n_tokens must be in [1, ld]", b);
    n_cache[b] = h_n_tokens[b] - 1;
    if (kv->lens_ub[b] + n_cache[b] + 1 > kv->max_len)
      return fail(SPADE_ECAPACITY, "request %d: %d cached + %d prompt tokens overflow max_len %d", b, kv->lens_ub[b],
                  h_n_tokens[b], kv->max_len);
  }
  hipError_t e = launch_prefill_batch(m, kv, B, d_tokens, ld, n_cache.data(), (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "prefill_batch");
  kv->verified = false;
  return SPADE_OK;
}

spade_status spade_softmax(const float* d_logits, int rows, int V, float temperature, float* d_probs,
                           void* stream) {
  if (!d_logits || !d_probs) return fail(SPADE_EINVAL, "null pointer");
  if (rows < 1 || V < 2) return fail(SPADE_EINVAL, "rows must be >= 1 and V >= 2");
  if (!(temperature > 0.f && std::isfinite(temperature)))
    return fail(SPADE_EINVAL, "temperature must be finite and > 0");
  hipError_t e = launch_softmax(d_logits, rows, V, 1.0f / temperature, d_probs, (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "softmax");
  return SPADE_OK;
}

spade_status spade_model_set_split_k(spade_model m, int splits) {
  if (!m) return fail(SPADE_EINVAL, "null model");
  if (splits != -1 && splits != 0 && splits != 2 && splits != 4) return fail(SPADE_EINVAL, "splits must be -1, 0, 2 or 4");
  m->split_ks = splits;
  return SPADE_OK;
}

spade_status spade_kv_commit(spade_kv kv, int B, const int32_t* d_n_accepted, const int32_t* d_correction,
                             void* stream) {
  if (!kv || !d_n_accepted || !d_correction) return fail(SPADE_EINVAL, "null pointer");
  if (!kv->verified) return fail(SPADE_EINVAL, "kv_commit needs a spade_verify on this cache since the last commit");
  if (B < 1 || B > kv->last_B) return fail(SPADE_EINVAL, "B=%d: the last spade_verify covered %d requests", B, kv->last_B);
  // the kernel clamps each k to [0, gamma] of that call, so the lengths grow
  // by at most gamma + 1
  hipError_t e = launch_commit(kv, B, kv->last_rows, d_n_accepted, d_correction, (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "kv_commit");
  for (int b = 0; b < B; ++b) kv->lens_ub[b] += kv->last_rows;
  kv->verified = false;
  return SPADE_OK;
}

spade_status spade_accept_from_logits(spade_model m, int B, int gamma, int V, const float* d_logits,
                                      const int32_t* d_draft_tokens, const float* d_draft_probs,
                                      const float* d_uniforms, const uint8_t* d_mode, float temperature,
                                      int32_t* d_n_accepted, int32_t* d_correction, void* stream) {
  if (!m || !d_logits || !d_mode || !d_n_accepted || !d_correction) return fail(SPADE_EINVAL, "null pointer");
  if (B < 1 || B > m->max_batch) return fail(SPADE_ECAPACITY, "B out of range");
  if (gamma < 0 || gamma + 1 > kMaxR) return fail(SPADE_ECAPACITY, "gamma out of range");
  if (gamma > 0 && !d_draft_tokens) return fail(SPADE_EINVAL, "draft tokens required when gamma > 0");
  if (V < 2) return fail(SPADE_EINVAL, "V must be >= 2");
  if (d_draft_probs && !d_uniforms) return fail(SPADE_EINVAL, "sampling needs uniforms");
  if (!(temperature > 0.f && std::isfinite(temperature)))
    return fail(SPADE_EINVAL, "temperature must be finite and > 0");
  AcceptCall ac{};
  ac.B = B;
  ac.gamma = gamma;
  ac.V = V;
  ac.logits = d_logits;
  ac.stats = nullptr;
  ac.drafts = d_draft_tokens;
  ac.q = d_draft_probs;
  ac.u = d_uniforms;
  ac.mode = d_mode;
  ac.inv_T = 1.0f / temperature;
  ac.n_out = d_n_accepted;
  ac.corr_out = d_correction;
  hipError_t e = launch_accept(m, ac, (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "accept_from_logits");
  return SPADE_OK;
}

spade_status spade_accept_from_logits_noalloc(int B, int gamma, int V, const float* d_logits,
                                              const int32_t* d_draft_tokens, const float* d_draft_probs,
                                              const float* d_uniforms, const uint8_t* d_mode, float temperature,
                                              int32_t* d_n_accepted, int32_t* d_correction, uint32_t* d_err,
                                              void* stream) {
  if (!d_logits || !d_mode || !d_n_accepted || !d_correction || !d_err) return fail(SPADE_EINVAL, "null pointer");
  if (B < 1 || B > kNoAllocMaxB)
    return fail(SPADE_ECAPACITY, "B=%d: the static scratch holds at most %d requests", B, kNoAllocMaxB);
  if (gamma < 0 || gamma + 1 > kMaxR) return fail(SPADE_ECAPACITY, "gamma out of range");
  if (gamma > 0 && !d_draft_tokens) return fail(SPADE_EINVAL, "draft tokens required when gamma > 0");
  if (V < 2) return fail(SPADE_EINVAL, "V must be >= 2");
  if (d_draft_probs && !d_uniforms) return fail(SPADE_EINVAL, "sampling needs uniforms");
  if (!(temperature > 0.f && std::isfinite(temperature)))
    return fail(SPADE_EINVAL, "temperature must be finite and > 0");
  AcceptCall ac{};
  ac.B = B;
  ac.gamma = gamma;
  ac.V = V;
  ac.logits = d_logits;
  ac.drafts = d_draft_tokens;
  ac.q = d_draft_probs;
  ac.u = d_uniforms;
  ac.mode = d_mode;
  ac.inv_T = 1.0f / temperature;
  ac.n_out = d_n_accepted;
  ac.corr_out = d_correction;
  hipError_t e = launch_accept_noalloc(ac, d_err, (hipStream_t)stream);
  if (e != hipSuccess) return hipfail(e, "accept_from_logits_noalloc");
  return SPADE_OK;
}

spade_status spade_profile_gemm(spade_model m, spade_kv kv, int kind, int B, int gamma, int launches,
                                void* stream) {
  if (!m || !kv) return fail(SPADE_EINVAL, "null pointer");
  if (kv->model != m) return fail(SPADE_EINVAL, "kv belongs to another model");
  if (kind < GEMM_QKV || kind > GEMM_LM) return fail(SPADE_EINVAL, "bad GEMM kind %d", kind);
  if (B < 1 || B > m->max_batch || B > kv->max_batch) return fail(SPADE_ECAPACITY, "B out of range");
  if (gamma < 0 || gamma > m->max_gamma) return fail(SPADE_ECAPACITY, "gamma out of range");
  if (launches < 1) return fail(SPADE_EINVAL, "launches must be >= 1");
  for (int b = 0; b < B; ++b)
    if (kv->lens_ub[b] + gamma + 1 > kv->max_len) return fail(SPADE_ECAPACITY, "KV capacity");
  const int R = gamma + 1;
  for (int i = 0; i < launches; ++i) {
    ForwardCall fc{};
    fc.b0 = 0;
    fc.nb = B;
    fc.R = R;
    fc.logits_out = m->ws.logits;
    fc.inv_T = 1.0f;
    hipError_t e = launch_layer_gemm(m, kv, kind, i % m->dims.L, fc, (hipStream_t)stream);
    if (e != hipSuccess) return hipfail(e, "profile_gemm");
  }
  return SPADE_OK;
}

spade_status spade_wide_tiling(int kind, int rows, int n_units, int k, int n_cu, int* row_tiles, int* panels,
                               int* k_splits) {
  if (!row_tiles || !panels || !k_splits) return fail(SPADE_EINVAL, "null pointer");
  if (kind < GEMM_QKV || kind > GEMM_LM || rows <= kWideMinRows || n_units < 1 || k < 256 || k % 256 != 0 ||
      n_cu < 1)
    return fail(SPADE_EINVAL, "shape out of range");
  const WideChoice c = wide_choice(kind, rows, n_units, k / 256, k, n_cu, 0, 0, 0, (size_t)-1, (size_t)-1);
  *row_tiles = c.rt;
  *panels = c.p;
  *k_splits = c.ks;
  return SPADE_OK;
}

spade_status spade_get_device_error(spade_model m, uint32_t* h_flags, void* stream) {
  if (!m || !h_flags) return fail(SPADE_EINVAL, "null pointer");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(h_flags, m->ws.err, 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemsetAsync(m->ws.err, 0, 4, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hipfail(e, "get_device_error");
  return SPADE_OK;
}

}  // extern "C"
