/*
 * dasc.h -- C ABI of the DASC state-checkpoint library for MI355X (gfx950).
 *
 * DASC ("Decay-Aware State Compression for Hybrid Linear-Attention Serving")
 * keeps only the long-horizon units of a gated delta-rule recurrent state in a
 * prefix-cache checkpoint, and on reuse either leaves the omitted units at zero
 * or refreshes them by replaying a bounded suffix.  This library implements
 * that path for one GPU:
 *
 *   dasc_plan     static selection plan from weight-derived decay (host only)
 *   dasc_pack     Store: ragged gather of retained units into checkpoint slots
 *   dasc_restore  Load:  scatter retained units back, omitted units = +0.0
 *   dasc_refresh  Load with refresh: replay the last W tokens of the gated
 *                 delta rule and overwrite only the omitted units
 *
 * State layout.  The paper writes a head state as S in R^{dv x dk} (Sec. 3.1,
 * Eq. 1).  This library stores its transpose S' = S^T as [dk, dv] fp32, dv
 * contiguous, so one KDA unit -- the key channel (h, k) of Sec. 4.1 -- is one
 * contiguous row of dv floats, and one GDN unit (a whole head) is dk such rows.
 * An active-state pool is [n_pool, L, H, dk, dv] fp32; a checkpoint pool is
 * [T, n_slots, C_rows, dv] fp32 (T = 1, C_rows = R for the flat layout).
 *
 * Conventions for every call.
 *   - Returns DASC_OK (0) or a negative DASC_E_* code; nothing throws or aborts.
 *   - Every argument the host can see is validated before any launch; a failed
 *     check returns an error and launches nothing.
 *   - The caller owns all memory.  The library allocates no device memory and
 *     keeps no state between calls, except the static device scratch array of
 *     dasc_refresh_noalloc (see there).
 *   - Device calls are asynchronous on the given stream and never synchronise.
 *     A NULL stream means the default (null) stream.
 *   - Indices that live in device memory (slot lists, row maps) cannot be seen
 *     by the host.  Kernels check each against its bound: a checkpoint whose
 *     slot index is out of range is skipped (nothing written for it), a packed
 *     row whose dense row is out of range is not written, and restore treats a
 *     dense row whose packed index is out of range as omitted (+0.0).
 *   - Device pointers to fp32 state/checkpoint data must be 16-byte aligned and
 *     dv must be a multiple of 4 (each row moves as 128-bit words).
 */
#ifndef DASC_H
#define DASC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
#define DASC_OK             0
#define DASC_E_INVAL       -1  /* null pointer, misalignment, scalar out of range */
#define DASC_E_SHAPE       -2  /* shape fields inconsistent with each other      */
#define DASC_E_WORKSPACE   -3  /* workspace smaller than dasc_refresh_workspace_bytes */
#define DASC_E_HIP         -4  /* the HIP runtime reported an error at launch    */
/* A device call first clears the calling thread's last HIP error (hipGetLastError), so
 * that DASC_E_HIP reports its own launches only: check HIP's state before the call if an
 * earlier error of the caller's matters.  Errors that happen while a kernel runs surface
 * at the caller's next synchronisation, as for any asynchronous launch. */
#define DASC_E_UNSUPPORTED -5  /* valid request with no kernel built for it      */
#define DASC_E_SCRATCH     -6  /* needs more than the static scratch of dasc_refresh_noalloc */

/* Longest replay window dasc_refresh accepts (tokens): keeps every per-head input
 * stream of a dk = 128 head within 1 GiB. */
#define DASC_MAX_WINDOW (1 << 21)

/* ---- enumerations -------------------------------------------------------- */
#define DASC_ARCH_KDA 0  /* channel-wise decay: unit = one (head, key channel) row */
#define DASC_ARCH_GDN 1  /* head-wise decay:    unit = one whole head              */

#define DASC_KEEP_THRESHOLD      0  /* keep u iff H_s(u) > W_max (Sec. 4.1)           */
#define DASC_KEEP_TOPK_PER_HEAD  1  /* keep the keep_k longest-horizon channels per head (KDA) */
#define DASC_KEEP_TOPK_PER_LAYER 2  /* keep the keep_k longest-horizon units per layer */

#define DASC_INIT_RESTORED 0  /* refresh replays from the restored active state      */
#define DASC_INIT_ZERO     1  /* refresh replays from a zero scratch state (Sec. 4.2) */

/* hipStream_t is `struct ihipStream_t *`; declared here so callers need no HIP headers. */
struct ihipStream_t;
typedef struct ihipStream_t *dasc_stream_t;

/* Shape of one recurrent state (all layers of one checkpoint). */
typedef struct dasc_shape {
  int32_t arch;        /* DASC_ARCH_KDA or DASC_ARCH_GDN                          */
  int32_t n_layers;    /* L: recurrent (linear-attention) layers                 */
  int32_t n_heads;     /* H: state (value) heads per layer                       */
  int32_t n_qk_heads;  /* Hqk: key heads per layer; value head j reads key head
                          j / (H / Hqk).  H % Hqk == 0.                          */
  int32_t dk;          /* key dimension: rows of a head state                    */
  int32_t dv;          /* value dimension: fp32 words per row, multiple of 4     */
} dasc_shape;

/* ---- plan (host only) ---------------------------------------------------- */

/* Static log-decay of Sec. 3.3, Eq. 2: g[i] = -exp(a_log[i]) * softplus(a + dt_bias[i]),
 * with softplus(x) = max(x, 0) + log1p(exp(-|x|)) in binary64.  The paper fixes the
 * input-dependent logit at a = -0.3.  dt_bias may be NULL (taken as 0).  Host arrays of
 * n doubles; g_out is written.  Errors: DASC_E_INVAL for NULL a_log/g_out or n < 0. */
int dasc_static_log_decay(const double *a_log, const double *dt_bias, double a, int64_t n,
                          double *g_out);

typedef struct dasc_plan_desc {
  dasc_shape shape;
  int32_t keep_mode;   /* DASC_KEEP_*                                             */
  int32_t keep_k;      /* units kept per head / per layer in the top-k modes      */
  int32_t w_max;       /* W_max (tokens), >= 0: threshold of Sec. 4.1 and upper
                          clamp of Eq. 7.  W_max = 0 keeps every unit ("dense").  */
  int32_t n_ranks;     /* T >= 1: TP degree for the per-rank slice table          */
  double eps;          /* epsilon of Eq. 3, in (0, 1); the paper uses 1e-3        */
  int64_t conv_bytes;  /* per-rank conv-state bytes per slot (Eq. 6 C_ckpt), >= 0 */
} dasc_plan_desc;

/* Plan outputs.  Array members are caller-owned HOST buffers whose sizes follow
 * from the shape alone (n_units_total = L*H*dk for KDA, L*H for GDN); a NULL
 * member is skipped.  Scalars are always written. */
typedef struct dasc_plan_out {
  uint8_t *keep;          /* [n_units_total] 1 = retained (global), 0 = omitted (local) */
  double *horizon;        /* [n_units_total] H_s = ln(eps) / g (Eq. 3)                  */
  int32_t *unit_count;    /* [L*H] retained units of each (layer, head)                 */
  int32_t *off;           /* [L*H+1] first packed row of each (layer, head); off[L*H] = R */
  int32_t *layer_off;     /* [L+1] App. B offsets o_l in units: o_0 = 0, o_{l+1} = o_l + r_l */
  int32_t *layer_off_rows; /* [L+1] the same offsets in packed rows (o_l * rows_per_unit): the
                              layer_off_rows argument of the padded layout (App. B Scheme 1) */
  int32_t *unit_row;      /* [L*H*dk] capacity: dense row (l*H + h)*dk + c of packed row j,
                             j < R, in (layer, head, channel) order                     */
  int32_t *inv_row;       /* [L*H*dk] packed row of each dense row, -1 if omitted       */
  int32_t *w_units;       /* [n_units_total] Eq. 7 window of each omitted unit, 0 if kept */
  int32_t *rank_begin;    /* [T+1] first packed row of each rank slice; rank_begin[T] = R */
  int64_t *send;          /* [T*T] send[o*T + s]: units computed on rank o (owner
                             floor(h*T/H)) that are stored in rank s's slice (Sec. 4.3) */
  int64_t n_rows;         /* R: packed rows per checkpoint                              */
  int64_t n_units;        /* retained units, sum_l r_l                                  */
  int32_t rows_per_unit;  /* 1 (KDA) or dk (GDN)                                        */
  int32_t w_replay;       /* Eq. 7: max window over omitted units, 0 if none            */
  int64_t slice_units;    /* C = ceil(n_units / T) (Sec. 4.3)                           */
  int64_t slice_rows;     /* C * rows_per_unit: rows of one rank slice                  */
  double c_temp_rag;      /* Eq. 6: sum_l n_l / sum_l r_l (inf if nothing retained)    */
  double c_temp_pad;      /* Sec. 4.1 padded layout: sum_l n_l / (L * R_max)            */
  double layout_gain;     /* R_max / r_bar (App. B)                                     */
  int64_t r_max_rows;     /* R_max * rows_per_unit: rows every layer reserves per checkpoint
                             in the padded layout (App. B Scheme 1)                     */
  double c_ckpt;          /* Eq. 6 C_ckpt with per-rank bottleneck: (dense/T + conv) /
                             (C * unit bytes + conv)                                    */
  int64_t slot_bytes_rank;       /* C * unit bytes + conv_bytes (Eq. 8 b_bottleneck)    */
  int64_t dense_slot_bytes_rank; /* ceil(n_units_total / T) * unit bytes + conv_bytes   */
} dasc_plan_out;

/* Build the static plan (Sec. 3.3, Sec. 4.1-4.3, App. B) from per-unit static
 * log-decay g_static (host, [L,H,dk] for KDA or [L,H] for GDN, every entry finite
 * and < 0).  Selection: DASC_KEEP_THRESHOLD keeps u iff H_s(u) > w_max (equality
 * omits); the top-k modes rank by H_s descending with ties to the lower unit index.
 * Pure host function: deterministic, bit-identical for identical inputs, no device use.
 * Errors: DASC_E_INVAL (NULL desc/g_static/out, eps not in (0,1), g not finite and
 * negative, w_max < 0, n_ranks < 1, keep_k out of range, conv_bytes < 0),
 * DASC_E_SHAPE (non-positive dims, H % Hqk != 0, per-head top-k on GDN,
 * L*H*dk >= 2^31). */
int dasc_plan(const dasc_plan_desc *desc, const double *g_static, dasc_plan_out *out);

/* App. C.1, Eq. 8: *slots = floor(budget_bytes / slot_bytes) - 1 (allocator slot 0 is
 * reserved).  Errors: DASC_E_INVAL if slots is NULL, budget_bytes < 0 or slot_bytes <= 0. */
int dasc_matched_slots(int64_t budget_bytes, int64_t slot_bytes, int64_t *slots);

/* Sec. 4.3, stage 1: a model-load-time permutation of linear-attention head bundles
 * across the T tensor-parallel ranks that lowers the retained rows of the most loaded
 * rank (which bounds the number of resident checkpoints).  Applying it to every
 * coupled weight and state tensor is an exact reindexing.  A bundle is one query/key
 * head with the H/Hqk value heads that share it; rank r computes bundle positions
 * [r*Hqk/T, (r+1)*Hqk/T) of every layer.  The paper gives no algorithm; this one
 * places bundles by retained rows, largest first (ties: lower layer, then lower
 * bundle), on the least loaded rank (ties: lower rank) that still has room in that
 * layer, keeps each rank's bundles in their original order, and returns the identity
 * whenever the result would be no better, so the worst rank never grows.
 *   unit_count: host int32 [L*H], retained units per (layer, head) as dasc_plan
 *     returns them (KDA: rows in [0, dk]; GDN: 0 or 1).
 *   head_perm: host int32 [L*H] out; head_perm[l*H + p] = original head at position p.
 *   rank_rows, rank_rows_identity: host int64 [T] out; retained rows per rank after
 *     the permutation and before it.
 * Errors: DASC_E_INVAL (NULL pointer, n_ranks < 1, Hqk % n_ranks != 0, a count out of
 * range), DASC_E_SHAPE (bad shape). */
int dasc_tp_permutation(const dasc_shape *shape, const int32_t *unit_count, int32_t n_ranks,
                        int32_t *head_perm, int64_t *rank_rows, int64_t *rank_rows_identity);

/* Static message for a status code (never NULL). */
const char *dasc_strerror(int code);

/* ---- Store: ragged pack (Sec. 4.1, App. B "Scheme 2") -------------------- */

/* For i < n and packed row j < n_rows:
 *     ckpt[r][dst_slot[i]][j - r*slice_rows][:] = states[src_slot[i]][unit_row[j]][:],
 *     r = j / slice_rows,
 * a bit-exact copy of dv fp32 words.  States are a pool [n_pool, L, H, dk, dv] whose
 * rows are addressed as [n_pool, L*H*dk, dv]; ckpt is [n_ranks, n_ckpt_slots,
 * slice_rows, dv].  n_ranks = 1 with slice_rows = n_rows is the flat layout
 * [n_ckpt_slots, R, dv]; n_ranks = T with slice_rows = the plan's slice_rows is the
 * per-rank slice layout of Sec. 4.3 (one device).  Checkpoint rows no packed row maps
 * to are not written.
 *   states, ckpt: device, 16-byte aligned.  src_slot, dst_slot: device int32 [n].
 *   unit_row: device int32 [n_rows] (dasc_plan's unit_row).
 * Errors: DASC_E_INVAL (NULL pointer with n > 0 and n_rows > 0, misalignment, n < 0,
 * n_pool < 1, n_ckpt_slots < 1, n_ranks < 1, slice_rows * n_ranks < n_rows),
 * DASC_E_SHAPE (bad shape, n_rows > L*H*dk, dv % 4 != 0), DASC_E_HIP. */
int dasc_pack(const dasc_shape *shape,
              const float *states, int64_t n_pool, const int32_t *src_slot,
              const int32_t *unit_row, int64_t n_rows,
              float *ckpt, int64_t n_ckpt_slots, const int32_t *dst_slot,
              int32_t n_ranks, int64_t slice_rows, int32_t n, dasc_stream_t stream);

/* ---- Load without refresh: restore with zero-fill (Sec. 4.2, DASC-NR) ----- */

/* For i < n and every dense row d < L*H*dk of the destination state:
 *     p = inv_row[d];
 *     states[dst_slot[i]][d][:] = (0 <= p < n_rows) ? ckpt[r][src_slot[i]][p - r*slice_rows][:]
 *                                                   : +0.0 (all bits clear),
 *     r = p / slice_rows.
 * Every row of every destination state is written (no separate memset needed).
 *   ckpt, states: device, 16-byte aligned.  inv_row: device int32 [L*H*dk]
 *   (dasc_plan's inv_row).  src_slot, dst_slot: device int32 [n].
 * Errors: as dasc_pack. */
int dasc_restore(const dasc_shape *shape,
                 const float *ckpt, int64_t n_ckpt_slots, const int32_t *src_slot,
                 int32_t n_ranks, int64_t slice_rows, int64_t n_rows,
                 const int32_t *inv_row,
                 float *states, int64_t n_pool, const int32_t *dst_slot,
                 int32_t n, dasc_stream_t stream);

/* ---- Padded checkpoints (App. B, Scheme 1: the comparison layout) --------- */

/* Store and Load with the padded layout: every layer reserves r_max_rows rows per
 * checkpoint (the largest layer's retained rows), ckpt = [L, n_ckpt_slots, r_max_rows,
 * dv]; entry e < r_l of layer l holds the e-th retained row of that layer, padding is
 * not written.  Same retained values as the ragged layout; it needs L * r_max_rows
 * rows per checkpoint instead of n_rows (the layout gain of Eq. 6).
 *   layer_off_rows: device int32 [L+1], dasc_plan's layer_off_rows.
 *   r_max_rows: dasc_plan's r_max_rows; rows a layer has past it are not written
 *     (pack) and restore as +0.0.
 *   Other arguments as dasc_pack / dasc_restore (flat addressing, no rank slices).
 * Errors: as dasc_pack / dasc_restore; DASC_E_INVAL also for r_max_rows < 1 with
 * n_rows > 0 or r_max_rows >= 2^31. */
int dasc_pack_padded(const dasc_shape *shape, const float *states, int64_t n_pool,
                     const int32_t *src_slot, const int32_t *unit_row, int64_t n_rows,
                     const int32_t *layer_off_rows, int64_t r_max_rows,
                     float *ckpt, int64_t n_ckpt_slots, const int32_t *dst_slot,
                     int32_t n, dasc_stream_t stream);

/* For every dense row d of layer l of each destination state:
 *     states[dst_slot[i]][d][:] = ckpt[l][src_slot[i]][inv_row[d] - layer_off_rows[l]][:]
 * when inv_row[d] >= 0 (and the entry lies in [0, r_max_rows)), else +0.0. */
int dasc_restore_padded(const dasc_shape *shape, const float *ckpt, int64_t n_ckpt_slots,
                        const int32_t *src_slot, const int32_t *layer_off_rows,
                        int64_t r_max_rows, int64_t n_rows, const int32_t *inv_row,
                        float *states, int64_t n_pool, const int32_t *dst_slot, int32_t n,
                        dasc_stream_t stream);

/* ---- INT8 checkpoints (App. E.1, Eq. 10) ---------------------------------- */

/* Pack with symmetric INT8 quantisation.  One scale per (layer, head, key channel),
 * shared over dv -- one scale per state row here: for packed row j of checkpoint i,
 *     a = max_v |x_v|,  s = max(a, 1e-8) / 127,  q_v = clip(rne(x_v / s), -127, 127),
 * with x = states[src_slot[i]][unit_row[j]][:], computed in FP32 with correctly rounded
 * divisions; q[dst_slot[i]][j][:] = q_v (int8), scale[dst_slot[i]][j] = s (FP32).
 *   states: device fp32 pool [n_pool, L*H*dk, dv], 16-byte aligned.
 *   q: device int8 [n_ckpt_slots, n_rows, dv], 4-byte aligned.
 *   scale: device fp32 [n_ckpt_slots, n_rows].
 *   unit_row: device int32 [n_rows]; src_slot, dst_slot: device int32 [n].
 * Flat layout only (no rank slices).  States must be finite.
 * Errors: as dasc_pack; DASC_E_UNSUPPORTED unless dv is a power of two in [4, 1024]. */
int dasc_pack_q8(const dasc_shape *shape, const float *states, int64_t n_pool,
                 const int32_t *src_slot, const int32_t *unit_row, int64_t n_rows,
                 int8_t *q, float *scale, int64_t n_ckpt_slots, const int32_t *dst_slot,
                 int32_t n, dasc_stream_t stream);

/* Restore from INT8 checkpoints: dequantise once into fresh FP32 active states,
 *     states[dst_slot[i]][d][:] = (0 <= p < n_rows) ? q[src_slot[i]][p][:] * scale[src_slot[i]][p]
 *                                                   : +0.0,    p = inv_row[d],
 * for every dense row d (the product is one FP32 multiply per element).
 * Arguments as dasc_pack_q8 / dasc_restore.  Errors: as dasc_pack_q8. */
int dasc_restore_q8(const dasc_shape *shape, const int8_t *q, const float *scale,
                    int64_t n_ckpt_slots, const int32_t *src_slot, int64_t n_rows,
                    const int32_t *inv_row, float *states, int64_t n_pool,
                    const int32_t *dst_slot, int32_t n, dasc_stream_t stream);

/* ---- Load with refresh: bounded-suffix replay (Sec. 4.2 DASC-WR, Eq. 1) --- */

/* Device workspace dasc_refresh and dasc_restore_refresh need for n_req requests and
 * window W.  GDN heads at dk = dv = 128 hold the state-independent factor of every
 * 32-token chunk there (the chunk's (I + A)^{-1} Diag(beta) of the WY form of Eq. 1,
 * split into two bf16 words per entry) between the two launches of their kernel:
 * n_req * n_heads * ceil(W / 32) * 4096 bytes.  Every other shape needs 0.  The caller
 * owns it; its contents need not be initialised and are dead after the call.
 * Errors: DASC_E_INVAL (NULL shape/bytes, n_req < 1, W < 1), DASC_E_SHAPE. */
int dasc_refresh_workspace_bytes(const dasc_shape *shape, int32_t n_req, int32_t W,
                                 size_t *bytes);

/* Replay the gated delta rule of Eq. 1 over the last W tokens for one layer and
 * overwrite only the omitted units, for each request i < n_req whose active state is
 * pool slot slot[i].  With S' = S^T (rows = key channels), per token t:
 *     S~  = Diag(exp(g_t)) S'_{t-1}
 *     S'_t = S~ + beta_t k_t (v_t - S~^T k_t)^T
 * S'_0 is the head's current (restored) state (DASC_INIT_RESTORED) or zero
 * (DASC_INIT_ZERO).  KDA: rows c with inv_row[(layer*H + h)*dk + c] < 0 receive
 * S'_W[c]; all other rows keep their bits.  GDN: a head is omitted when its rows are,
 * and its whole state receives S'_W.  Heads with nothing omitted are not touched.
 *   inv_row: device int32 [L*H*dk] (dasc_plan's inv_row; only the sign is read).
 *   states:  device fp32 pool [n_pool, L, H, dk, dv], 16-byte aligned, read and written.
 *   slot:    device int32 [n_req].
 *   k:    device bf16 bits [n_req, Hqk, W, dk]   (16-byte aligned, dk % 8 == 0)
 *   v:    device bf16 bits [n_req, H,   W, dv]   (16-byte aligned)
 *   g:    device fp32 log-gates, [n_req, H, W, dk] (KDA) or [n_req, H, W] (GDN)
 *   beta: device fp32 [n_req, H, W]
 *   workspace: device, at least dasc_refresh_workspace_bytes, 16-byte aligned (may be
 *              NULL if that is 0); overlapping calls must not share one.
 * Precision.  The state is fp32 and bf16 inputs are widened exactly.  At dk = dv = 128 the
 * chunked WY form of Eq. 1 runs on bf16 matrix cores: every fp32 operand of a product is
 * split into bf16 high and low parts and the product is the sum of three bf16 products
 * (hi*hi + hi*lo + lo*hi) accumulated in fp32, about 16 significant bits per term; and
 * each per-token log-gate is floored at -10 (a decay of at least 4.5e-5 per token, which
 * keeps the factorised decays finite; it changes the state by at most 4.5e-5 of its
 * magnitude per floored token).  Other shapes run a plain fp32 per-token recurrence with
 * no floor.  Measured against an fp64 replay: within 2e-3 of each head's largest
 * refreshed magnitude (about 1e-5 at the shapes of Sec. 5.1).
 * Errors: DASC_E_INVAL (NULL pointer, misalignment, layer out of [0, L), n_req < 1,
 * W < 1 or W > DASC_MAX_WINDOW, bad init_mode, n_pool < 1), DASC_E_SHAPE (bad shape),
 * DASC_E_WORKSPACE, DASC_E_UNSUPPORTED (dk not in {16, 32, 64, 128} or dv > 256),
 * DASC_E_HIP. */
int dasc_refresh(const dasc_shape *shape, int32_t layer, const int32_t *inv_row,
                 float *states, int64_t n_pool, const int32_t *slot,
                 const uint16_t *k, const uint16_t *v, const float *g, const float *beta,
                 int32_t n_req, int32_t W, int32_t init_mode,
                 void *workspace, size_t workspace_bytes, dasc_stream_t stream);

/* ---- Load with refresh, allocating nothing -------------------------------- */

/* Size of the device scratch array dasc_refresh_noalloc uses in place of a workspace
 * (64 MiB per device: the GDN factor records of, for example, 16 requests x 32 heads at
 * W = 1024, or 8 requests x 32 heads at W = 2048). */
#define DASC_NOALLOC_SCRATCH_BYTES (64ll << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): dasc_refresh with no workspace
 * argument.  The scratch dasc_refresh would take from the workspace (the GDN factor
 * records, dasc_refresh_workspace_bytes of them) lives in a device array inside the
 * library, DASC_NOALLOC_SCRATCH_BYTES on each device it runs on, held until the process
 * ends; its device address is looked up once per device, on the first call with that
 * device current.  The call allocates nothing (no hipMalloc, no allocating library
 * routine).  Arguments, layouts, results and precision are those of dasc_refresh; the
 * kernels are the same, so the results are bit-identical to dasc_refresh's.
 * Every call on one device shares that device's array: calls that overlap on one device
 * (different streams, or threads without ordering) race and must not be issued.  The
 * stream must belong to the current device.
 * Errors: those of dasc_refresh (without DASC_E_WORKSPACE); DASC_E_SCRATCH, before
 * anything is launched, when dasc_refresh_workspace_bytes for this shape, n_req and W
 * exceeds DASC_NOALLOC_SCRATCH_BYTES; DASC_E_HIP if the array's address cannot be found. */
int dasc_refresh_noalloc(const dasc_shape *shape, int32_t layer, const int32_t *inv_row,
                         float *states, int64_t n_pool, const int32_t *slot,
                         const uint16_t *k, const uint16_t *v, const float *g, const float *beta,
                         int32_t n_req, int32_t W, int32_t init_mode, dasc_stream_t stream);

/* ---- Load with refresh, fused (Sec. 4.2: restore, then DASC-WR) ----------- */

/* What dasc_restore followed by dasc_refresh does for one layer, without the separate
 * restore pass (one launch for KDA heads; GDN heads take two, the state-independent
 * factor launch of dasc_refresh and then the fused recurrence):
 * for each request i < n_req, the rows of layer `layer` of states[dst_slot[i]] receive
 *   - omitted rows of heads that have any (KDA rows; GDN whole heads): S'_W of the
 *     replay above, started from the restored head (kept rows taken from checkpoint
 *     src_slot[i], omitted rows +0.0) or from zero (DASC_INIT_ZERO);
 *   - every other row: its packed row of checkpoint src_slot[i], bit for bit (+0.0 if
 *     inv_row points outside [0, n_rows)).
 * The state is read from the checkpoint, never from `states`; every row of the layer
 * is written once and rows of other layers are not touched.  The result equals
 * dasc_restore (of this layer) followed by dasc_refresh bit for bit.
 *   ckpt, n_ckpt_slots, n_ranks, slice_rows, n_rows, inv_row: as in dasc_restore.
 *   src_slot: device int32 [n_req], checkpoint slot per request.
 *   states, dst_slot: as states, slot in dasc_refresh (the pool need not hold the
 *   restored state beforehand).
 *   k, v, g, beta, W, init_mode, workspace: as in dasc_refresh.
 * Built for dk = dv = 128 (the shapes of Sec. 5.1); precision as in dasc_refresh.
 * Errors: those of dasc_restore and dasc_refresh; DASC_E_UNSUPPORTED unless
 * dk = dv = 128. */
int dasc_restore_refresh(const dasc_shape *shape, int32_t layer,
                         const float *ckpt, int64_t n_ckpt_slots, const int32_t *src_slot,
                         int32_t n_ranks, int64_t slice_rows, int64_t n_rows,
                         const int32_t *inv_row, float *states, int64_t n_pool,
                         const int32_t *dst_slot,
                         const uint16_t *k, const uint16_t *v, const float *g, const float *beta,
                         int32_t n_req, int32_t W, int32_t init_mode,
                         void *workspace, size_t workspace_bytes, dasc_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DASC_H */
