// Accept / reject and the correction draw for one request (Sec. III-C;
// Algorithm 1, the verify / accept / sample / correct steps), run by one
// workgroup of NT threads (COH: logits and LM-head statistics are read with
// sc1 loads, for a caller whose other workgroups wrote them in the same
// launch).
#pragma once

#include "device_util.h"

namespace spade {

struct AcceptParams {
  const float* logits;
  const float* stats;
  int NU;
  int panels;  // 0: stats holds NU workgroup entries per row; > 0: one entry per panel
  int B, V, gamma, R;
  const int32_t* drafts;
  const float* q;
  const float* u;
  const uint8_t* mode;
  float inv_T;
  int32_t* n_out;
  int32_t* corr_out;
  uint32_t* err;
  // > 0: the correction draws of sampling requests are left to
  // correct_slices over this many vocabulary slices (accept_request stores
  // the log-sum-exp of the draw's row in corr_lse[b]); corr_part /
  // corr_cnt: per-slice winners and per-request arrival counters
  int corr_slices;
  float* corr_lse;
  float* corr_part;
  uint32_t* corr_cnt;
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

struct Best {
  float s;
  int a;
};

__device__ __forceinline__ Best better(Best x, Best y) {
  if (y.s > x.s || (y.s == x.s && y.a < x.a)) return y;
  return x;
}

template <bool COH>
__device__ __forceinline__ float ld_any(const float* p) {
  if constexpr (COH) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else return *p;
}

// Gumbel-max scores of token v for the correction draw: the residual
// max(0, p - q) (log w + g, -inf where w <= 0) and p itself (z + g), with z
// the logit over the temperature and g the token's Gumbel noise.  No
// contraction, so every caller gets the same roundings.
__device__ __forceinline__ float corr_score_p(float logit, float invT, float g) {
#pragma clang fp contract(off)
  const float z = logit * invT;
  return z + g;
}

__device__ __forceinline__ float corr_score_res(float logit, float invT, float lse, float qv, float g) {
#pragma clang fp contract(off)
  const float z = logit * invT;
  const float w = expf(z - lse) - qv;
  return w > 0.f ? logf(w) + g : -INFINITY;
}

// Whether request b draws by sampling (else greedily); the accept step and
// the sliced correction decide it the same way.
__device__ __forceinline__ bool accept_samples(const AcceptParams& p, int b) {
  return p.mode[b] == SPADE_SAMPLE && p.u != nullptr && (p.gamma == 0 || p.q != nullptr);
}

struct AcceptSmem {
  float rlse[kMaxR];
  int rarg[kMaxR];
  int x[kMaxR];                     // draft tokens (clamped)
  float lx[kMaxR], qx[kMaxR], ux[kMaxR];  // sampling: logit and q at the draft, its uniform
  Best bpart[16];
  int n_s;
};

template <int NT, bool COH>
__device__ __forceinline__ void accept_request(const AcceptParams& p, int b, AcceptSmem& sm) {
  constexpr int NWV = NT / 64;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int R = p.R, V = p.V, G = p.gamma;

  const bool sample = accept_samples(p, b);
  if (!sample && p.mode[b] == SPADE_SAMPLE && tid == 0) flag_error(p.err, SPADE_DERR_NOQ);
  const float invT = sample ? p.inv_T : 1.0f;
  const float* lg = p.logits + (size_t)b * R * V;

  // the drafts and what the accept chain reads for them, one thread per draft
  if (tid < G) {
    int x = p.drafts[(size_t)b * G + tid];
    if (x < 0 || x >= V) {
      flag_error(p.err, SPADE_DERR_TOKEN);
      x = x < 0 ? 0 : V - 1;
    }
    sm.x[tid] = x;
    if (sample) {
      sm.lx[tid] = ld_any<COH>(lg + (size_t)tid * V + x);
      sm.qx[tid] = p.q[((size_t)b * G + tid) * V + x];
      sm.ux[tid] = p.u[(size_t)b * (G + 1) + tid];
    }
  }

  // row statistics over the vocabulary: wave r merges row r from the LM
  // head's per-workgroup partials (or, without them, from the logits), in a
  // fixed order
  for (int r = wave; r < R; r += NWV) {
    RowStat st{-INFINITY, 0.f, 0x7fffffff};
    if (p.stats != nullptr && p.panels > 0) {
      // per-panel statistics: rebuild the NU workgroup entries of the skinny
      // LM head (workgroup q folds panels q, q + NU, ... in order), then merge
      // them exactly as below
      // (the panels of an entry are requested sixteen at a time and then
      // folded in order, so the loads do not wait for one another)
      constexpr int kBatch = 16;
      const float* sp = p.stats + (size_t)(b * R + r) * p.panels * 3;
      for (int q = lane; q < p.NU; q += 64) {
        RowStat one{-INFINITY, 0.f, 0x7fffffff};
        for (int u0 = q; u0 < p.panels; u0 += kBatch * p.NU) {
          RowStat ps[kBatch];
#pragma unroll
          for (int j = 0; j < kBatch; ++j) {
            const int u = u0 + j * p.NU;
            ps[j] = RowStat{-INFINITY, 0.f, 0x7fffffff};
            if (u < p.panels)
              ps[j] = RowStat{ld_any<COH>(sp + u * 3), ld_any<COH>(sp + u * 3 + 1),
                              __float_as_int(ld_any<COH>(sp + u * 3 + 2))};
          }
#pragma unroll
          for (int j = 0; j < kBatch; ++j)
            if (ps[j].m != -INFINITY) one = merge_stat(one, ps[j]);
        }
        if (one.m != -INFINITY) st = merge_stat(st, one);
      }
    } else if (p.stats != nullptr) {
      const float* sp = p.stats + (size_t)(b * R + r) * p.NU * 3;
#pragma unroll 8
      for (int q = lane; q < p.NU; q += 64) {
        const RowStat one{ld_any<COH>(sp + q * 3), ld_any<COH>(sp + q * 3 + 1),
                          __float_as_int(ld_any<COH>(sp + q * 3 + 2))};
        if (one.m != -INFINITY) st = merge_stat(st, one);
      }
    } else {
#pragma unroll 8
      for (int v = lane; v < V; v += 64) {
        const float z = ld_any<COH>(lg + (size_t)r * V + v) * invT;
        if (z != z) continue;
        st = merge_stat(st, RowStat{z, 1.f, v});
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      RowStat o;
      o.m = __shfl_xor(st.m, off);
      o.s = __shfl_xor(st.s, off);
      o.a = __shfl_xor(st.a, off);
      st = (lane & off) ? merge_stat(o, st) : merge_stat(st, o);
    }
    if (lane == 0) {
      sm.rlse[r] = st.m + logf(st.s);
      sm.rarg[r] = st.a;
    }
  }
  __syncthreads();

  if (tid == 0) {
    int n = G;
    for (int i = 0; i < G; ++i) {
      bool ok;
      if (!sample) {
        ok = (sm.x[i] == sm.rarg[i]);
      } else {
        const float px = expf(sm.lx[i] * invT - sm.rlse[i]);
        ok = sm.ux[i] * sm.qx[i] < px;
      }
      if (!ok) {
        n = i;
        break;
      }
    }
    sm.n_s = n;
  }
  __syncthreads();
  const int n = sm.n_s;
  int corr = 0;
  if (!sample) {
    corr = sm.rarg[n];
  } else if (p.corr_slices > 0) {
    // correct_slices draws it after this launch; its arrival counter starts
    // that launch at zero
    if (tid == 0) {
      p.corr_lse[b] = sm.rlse[n];
      p.n_out[b] = n;
      p.corr_cnt[b] = 0u;
    }
    return;
  } else {
    const uint64_t seed = (uint64_t)__float_as_uint(p.u[(size_t)b * (G + 1) + G]);
    const float* row = lg + (size_t)n * V;
    const bool residual = n < G;
    const float* qrow = residual ? p.q + ((size_t)b * G + n) * V : nullptr;
    const float lse = sm.rlse[n];
    for (int pass = 0; pass < 2; ++pass) {
      const bool use_res = residual && pass == 0;
      Best bst{-INFINITY, 0x7fffffff};
#pragma unroll 4
      for (int v = tid; v < V; v += NT) {
        const float lv = ld_any<COH>(row + v), g = gumbel_at(seed, v);
        const float sc = use_res ? corr_score_res(lv, invT, lse, qrow[v], g) : corr_score_p(lv, invT, g);
        if (sc != sc) continue;
        bst = better(bst, Best{sc, v});
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const Best o{__shfl_xor(bst.s, off), __shfl_xor(bst.a, off)};
        bst = better(bst, o);
      }
      if (lane == 0) sm.bpart[wave] = bst;
      __syncthreads();
      Best t = sm.bpart[0];
      for (int w = 1; w < NWV; ++w) t = better(t, sm.bpart[w]);
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

__device__ __forceinline__ Best wave_best(Best x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = better(x, Best{__shfl_xor(x.s, off), __shfl_xor(x.a, off)});
  return x;
}

// Slice s of corr_slices of the correction draw of a sampling request b,
// after accept_request (previous launch) stored n and the row's log-sum-exp:
// the best residual score and the best score under p over the slice's tokens
// (NaN scores skipped, as in the one-workgroup draw), published write-through;
// the last slice to arrive takes the best of all slices (the order of this
// maximum does not matter: ties go to the lower token id) and stores the
// correction, the residual's winner unless the residual had no mass.
// NT threads, one workgroup per (slice, request).
template <int NT>
__device__ __forceinline__ void correct_slice(const AcceptParams& p, int b, int s) {
  constexpr int NWV = NT / 64;
  __shared__ Best sres[NWV], sp[NWV];
  __shared__ int last;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (!accept_samples(p, b)) return;  // uniform
  const int V = p.V, G = p.gamma, S = p.corr_slices;
  const int n = p.n_out[b];
  const bool residual = n < G;
  const float invT = p.inv_T, lse = p.corr_lse[b];
  const uint64_t seed = (uint64_t)__float_as_uint(p.u[(size_t)b * (G + 1) + G]);
  const float* row = p.logits + ((size_t)b * (G + 1) + n) * V;
  const float* qrow = residual ? p.q + ((size_t)b * G + n) * V : nullptr;
  const int per = (V + S - 1) / S;
  const int v0 = s * per, v1 = min(V, v0 + per);
  Best br{-INFINITY, 0x7fffffff}, bp{-INFINITY, 0x7fffffff};
#pragma unroll 4
  for (int v = v0 + tid; v < v1; v += NT) {
    const float lv = row[v], g = gumbel_at(seed, v);
    const float sc = corr_score_p(lv, invT, g);
    if (sc == sc) bp = better(bp, Best{sc, v});
    if (residual) {
      const float sr = corr_score_res(lv, invT, lse, qrow[v], g);
      if (sr == sr) br = better(br, Best{sr, v});
    }
  }
  br = wave_best(br);
  bp = wave_best(bp);
  if (lane == 0) {
    sres[wave] = br;
    sp[wave] = bp;
  }
  __syncthreads();
  const Rsrc rp = make_rsrc(p.corr_part, (uint32_t)(p.B * kCorrMaxSlices * 4 * 4));
  const uint32_t base = (uint32_t)((b * kCorrMaxSlices + s) * 4) * 4u;
  if (tid == 0) {
    for (int w = 1; w < NWV; ++w) {
      br = better(br, sres[w]);
      bp = better(bp, sp[w]);
    }
    st_f32<true>(rp, base, br.s);
    st_f32<true>(rp, base + 4u, __int_as_float(br.a));
    st_f32<true>(rp, base + 8u, bp.s);
    st_f32<true>(rp, base + 12u, __int_as_float(bp.a));
    __builtin_amdgcn_s_waitcnt(0);  // the winners have landed: arrive
    const uint32_t old = __hip_atomic_fetch_add(p.corr_cnt + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = old == (uint32_t)S - 1u;
    if (last) __hip_atomic_store(p.corr_cnt + b, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last || wave != 0) return;
  Best r{-INFINITY, 0x7fffffff}, q{-INFINITY, 0x7fffffff};
  for (int i = lane; i < S; i += 64) {
    const uint32_t off = (uint32_t)((b * kCorrMaxSlices + i) * 4) * 4u;
    r = better(r, Best{ld_f32<true>(rp, off), __float_as_int(ld_f32<true>(rp, off + 4u))});
    q = better(q, Best{ld_f32<true>(rp, off + 8u), __float_as_int(ld_f32<true>(rp, off + 12u))});
  }
  r = wave_best(r);
  q = wave_best(q);
  if (lane == 0) {
    int corr = q.a;
    if (residual) {
      if (r.s != -INFINITY) corr = r.a;
      else flag_error(p.err, SPADE_DERR_RESIDUAL);
    }
    p.corr_out[b] = corr;
  }
}

}  // namespace spade
