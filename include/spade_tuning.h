/*
 * spade_tuning.h -- schedule controls and measurement hooks of the
 * speculative-verify library (libspade.so), separate from the calls of the
 * method in spade.h.
 *
 * Every setter below changes how spade_verify schedules its kernels, never
 * what it computes: each setting gives bit-for-bit the same logits,
 * n_accepted and corrections (the tests force every setting and compare).
 * The defaults are chosen per call from the shape; a setter fixes or turns
 * off one choice, for measurement and for those tests.  Conventions as in
 * spade.h.
 */
#ifndef SPADE_TUNING_H
#define SPADE_TUNING_H

#include "spade.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Tiling of the batched projections.  A verify call with more than 16 rows
 * (B * (gamma + 1) > 16) and bf16 weights runs the QKV, O, gate/up and down
 * projections on the wide-row GEMM: each weight tile is read once per launch
 * and multiplied with `row_tiles` 16-row tiles of the activations held in
 * LDS; each wave owns `panels` 16-column weight panels, so that every
 * activation fragment read from LDS feeds that many matrix instructions.  The
 * row groups of one set of panels run on one XCD and share its L2.
 * row_tiles = 0 and panels = 0 (the defaults) are chosen per launch from the
 * shape and the compute-unit count; row_tiles 1..3 and panels 1..2 fix them
 * (the O and down projections, which can be k-split, take two panels per
 * wave with at most two row tiles and fall back to one tile and one panel);
 * row_tiles = -1 turns the wide-row GEMM off (the skinny engine then runs
 * once per 32 rows and streams the weights once per launch).  Results are
 * bit-for-bit the same under every setting: a row's dot products are summed
 * over the same k-ranges in the same order whatever the tiling.  Other values
 * return SPADE_EINVAL. */
spade_status spade_model_set_wide_tiles(spade_model m, int row_tiles, int panels);

/* Merge of the verify attention's chunk partials (bf16 cache, head_dim 128:
 * one workgroup per 256-key chunk of a (request, head), each giving a partial
 * -- row max, row sum, unnormalised output -- merged in chunk order).  mode 1: the last workgroup of a
 * (request, head) to finish merges its chunks, which makes every chunk
 * workgroup wait for its stores and an arrival counter; mode 2: the chunk
 * workgroups store their partials and exit, and a second launch merges each
 * (request, head); mode 0 (the default) chooses per call (mode 2 from four
 * chunks per compute unit).  Results are bit-for-bit the same under every
 * mode.  Other values return SPADE_EINVAL. */
spade_status spade_model_set_attn_merge(spade_model m, int mode);

/* Where the correction draw of a sampling request runs (Sec. III-C: sample
 * from norm(max(0, p - q)), or from p when every draft is accepted; the draw
 * is a Gumbel-max pass over the vocabulary).  mode 0 (the default) or 2: when
 * the call may sample (uniforms given, and draft_probs given or gamma = 0),
 * spade_verify (per-stage path) and spade_accept_from_logits run it in a
 * second launch over slices of 1024 tokens (at most 256 slices), one
 * workgroup per (slice, request), the last slice of a request to finish
 * taking the best of the slices; mode 1 keeps it in the request's accept
 * workgroup.  The single-launch pass always keeps it there.  Results are bit-for-bit the same under
 * every mode.  Other values return SPADE_EINVAL. */
spade_status spade_model_set_correction_slices(spade_model m, int mode);

/* Grouped-query attention chunks.  For a model with G = heads / K/V heads
 * > 1, when the attention partials are merged in a second launch (see
 * spade_model_set_attn_merge) and the G (gamma+1) rows of a request fit 48
 * rows, mode 0 (the default) computes each 256-key chunk for all G query
 * heads of a K/V head in one workgroup (the rows packed into 16-row MFMA
 * tiles), so the chunk's keys and values pass through a compute unit once;
 * mode 1 keeps one workgroup per query head.  Results are bit-for-bit the
 * same under both modes.  Other values return SPADE_EINVAL. */
spade_status spade_model_set_attn_grouped(spade_model m, int mode);

/* Prompt rows per request of a prefill forward (spade_prefill,
 * spade_prefill_batch; Sec. III-A: the context is run through the verifier
 * once before the first verification).  With a bf16 cache and head_dim 128,
 * rows = 0 (the default) lets a forward take as many prompt rows as the
 * workspace holds (up to 2048 rows in all), so the projections multiply each
 * weight tile with thousands of rows and run at matrix-core speed, and the
 * attention of rows past the first 16 runs on the prefill attention kernel
 * (16-row tiles, each computed as a verify call of its own); rows > 0 caps
 * the rows per request (at most 16: the verify attention kernels, 16 rows
 * per forward).  Other caches always take 16.  The cache contents, and so
 * every later result, are bit-for-bit the same under every setting.  rows < 0
 * returns SPADE_EINVAL. */
spade_status spade_model_set_prefill_rows(spade_model m, int rows);

/* Projection GEMM of forwards with many rows (prefill: hundreds to thousands
 * of prompt rows; bf16 weights).  A workgroup of eight waves owns 128 rows and
 * 256 columns and runs the k-loop in 32-k steps: the activations' step
 * through an LDS ring filled by direct loads, the weights' straight into
 * registers, so each weight byte is multiplied with 128 rows and each
 * activation byte read from LDS with 256 columns.  mode 0 (the default) uses
 * it for the QKV, O, gate/up and down projections once a launch has at least
 * one such workgroup per compute unit; mode 1 turns it off (the wide-row GEMM
 * runs instead); mode 2 uses it for every launch of more than 16 rows but
 * the LM head.  Results are bit-for-bit the same under every mode.  Other
 * values return SPADE_EINVAL. */
spade_status spade_model_set_big_gemm(spade_model m, int mode);

/* Projection GEMM of batched verification calls of up to 144 rows (e.g. 16
 * requests of gamma + 1 = 9 rows; bf16 weights).  A workgroup of eight waves
 * owns every row of the call and 256 columns, so each weight byte enters one
 * compute unit once per launch; the k-loop runs in 32-k steps with the
 * activations' step in an LDS ring filled by direct loads and the weights'
 * straight into registers.  The k-loop is split over 1-8 workgroups per
 * panel group (whole k-ranges of the eight); each stores its sums in the
 * workspace, and a second launch, one workgroup per panel group and 16-row
 * tile, adds them in range order and runs the epilogue.  mode 0 (the
 * default) uses it where it measured faster than the wide-row GEMM: the
 * gate/up projection of 113 to 144 rows, the O projection of 129 to 144, the
 * down projection of 137 to 144; mode 1 turns it off (the wide-row GEMM runs
 * instead); mode 2 uses it for every QKV, O, gate/up and down launch of 17
 * to 144 rows.  k_splits 0 chooses the split count per launch, 1..8 fixes
 * it.  Results are bit-for-bit the same under every setting.  Other values
 * return SPADE_EINVAL. */
spade_status spade_model_set_mid_gemm(spade_model m, int mode, int k_splits);

/* K splitting of the batched O and down projections on the wide-row GEMM.
 * Their weights have few panels (d_model / 16), so one workgroup per panel
 * group leaves most compute units idle; with `splits` = 2 or 4 each
 * workgroup streams only 1/splits of the k-blocks (whole k-ranges of the
 * engine's eight), publishes its partial sums to the workspace, and the
 * last workgroup of a panel group to finish adds them in range order and
 * runs the epilogue.  splits = 0 (the default) chooses per launch from the
 * shape, 1 turns k-splitting off, 2 or 4 fix it (falling back to 1 where the
 * workspace's published-value buffers are too small).  Results are
 * bit-for-bit the same under every setting.  Other values return
 * SPADE_EINVAL. */
spade_status spade_model_set_wide_k_splits(spade_model m, int splits);

/* K splitting of the small-batch projections.  A verify call with at most 16
 * rows and bf16 weights whose activation operand is too long for one LDS copy
 * (the 7B-shaped down projection, every projection of the 13B shape) runs the
 * QKV, O, gate/up or down projection split along K into `splits` parts: a
 * workgroup copies only its part of the operand into LDS and streams one
 * k-range of each of its panels; the last workgroup of a panel group to finish
 * completes the sums and runs the epilogue.  splits = 0 (the default) picks 2
 * or 4, the fewest whose part fits; 2 or 4 fix it (also where the whole
 * operand would fit) where the part fits; -1 turns it off (the operand is then
 * fetched from L2 with every weight tile).  Results are bit-for-bit the same
 * under every setting: each dot product is summed over the same eight k-ranges
 * in the same order.  Other values return SPADE_EINVAL. */
spade_status spade_model_set_split_k(spade_model m, int splits);

/* Measurement hook: launch the GEMM kernel of one projection alone, exactly
 * as spade_verify launches it for B requests of gamma drafts, `launches`
 * times (layer = i mod n_layers), on the workspace's current operands.
 * kind: 0 QKV (+RoPE, KV append), 1 O (+residual), 2 gate/up (+SiLU),
 * 3 down (+residual), 4 LM head.  It overwrites workspace activations and
 * cache rows past lens, so run it between verify calls, not inside a round. */
spade_status spade_profile_gemm(spade_model m, spade_kv kv, int kind, int B, int gamma, int launches,
                                void* stream);

/* Inspection hook (host only, no device): the tiling the wide-row GEMM picks
 * for a bf16 projection launch of `rows` rows (> 16), `n_units` 16-row weight
 * panels and `k` inputs (a multiple of 256) on `n_cu` compute units, with
 * every setting at its default and buffers large enough for any k-split.
 * kind as for spade_profile_gemm.  Writes the 16-row tiles per workgroup,
 * the panels per wave and the k-splits; SPADE_EINVAL on a null pointer or
 * a shape out of range. */
spade_status spade_wide_tiling(int kind, int rows, int n_units, int k, int n_cu, int* row_tiles, int* panels,
                               int* k_splits);

#ifdef __cplusplus
}
#endif

#endif /* SPADE_TUNING_H */
