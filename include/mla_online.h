/*
 * mla_online.h -- C ABI of the MLA-Online step of RedKnot-MLA (arXiv 2609.07008)
 * for AMD Instinct MI355X (gfx950).
 *
 * The step recomputes, at serving time, the part of a multi-head-latent-attention
 * layer that cannot be reused from per-document offline artifacts (Sec. 2.3,
 * Alg. 2):
 *   1. query-side RoPE relocation: each query is rotated into a document's
 *      canonical frame, R(t - p_s), instead of rewriting cached keys (eq:rope);
 *   2. absorbed-MLA attention over the single packed latent stream (d_c latent
 *      plus d_r decoupled RoPE key per token), one document segment (or one run
 *      of segments) at a time: Global heads on every row, Local heads only on
 *      protected rows (SelectiveMLA);
 *   3. a stable segmented log-sum-exp merge of the per-segment partials;
 *   4. the group-aligned sliced first output projection W_a, with the offline
 *      Local-head artifact z_off added on unprotected rows and replaced (never
 *      added) on protected rows (RestoreAndReplace, eq:factorization).
 * Beside the step the library exports the offline producer of the artifact
 * (Alg. 1), the protected token-row set (eq:protected), the shared second
 * projection y = W_b z and the adaptive MoE fanout (eq:moe).
 *
 * Conventions (all entry points):
 *  - Host arrays are read during the call only.  Device arrays are owned by the
 *    caller; the library allocates no device memory of its own beyond one
 *    fixed scratch array per GPU used only by mla_online_attend_planned_noalloc
 *    (everything else takes a caller-provided workspace) and keeps no per-call
 *    state.
 *  - All device work is enqueued on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream) in call order.  The host-plan attend,
 *    producer, protected-set and mla_online_plan calls copy a plan (segment
 *    tables and, for the first three, the work list) from a library-owned
 *    pinned host buffer of two slots per device on the same stream; reusing a
 *    slot waits for the copy that last read it, so a third back-to-back call
 *    may block the host until the first call's copy has run.  Every other
 *    call only enqueues kernels and never blocks.
 *  - HIP graph capture: the merge, o-proj, W_b, MoE and the planned
 *    protected-set, attend and o-proj calls enqueue kernels only (no memset or
 *    memcpy nodes) and may be captured.  The calls that upload a plan return MLA_ERR_UNSUPPORTED on a
 *    capturing stream, before enqueueing anything: their staging buffer is
 *    reused by later calls, so a replay would not read the captured plan.
 *  - Every entry point validates its arguments on the host before enqueueing
 *    anything and returns a status; it never aborts and never falls back to a
 *    different computation.  mla_last_error_detail() describes the last failure
 *    of the calling thread.
 *  - Layouts are dense row-major.  "bf16" is IEEE bfloat16 (uint16 storage).
 *    Device pointers to bf16 or float data must be 16-byte aligned.
 *  - Supported (d_latent, d_rope): (512, 64) -- the DeepSeek latent row of the
 *    paper's profiles -- and (64, 16).  Others return MLA_ERR_UNSUPPORTED.
 *
 * Notation: N request rows; a row r is also KV row r (storage order); H heads in
 * G output groups of hpg = H/G heads with one Global head per group (Sec. 3.1);
 * L_h = G*(hpg-1) Local heads per protected row; P protected rows; D = d_c+d_r.
 */
#ifndef MLA_ONLINE_H
#define MLA_ONLINE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum mla_status {
  MLA_OK = 0,
  MLA_ERR_NULL = 1,         /* a required pointer is NULL                           */
  MLA_ERR_SHAPE = 2,        /* inconsistent sizes, alignment or geometry            */
  MLA_ERR_UNSUPPORTED = 3,  /* valid but not built (head dims, group counts)        */
  MLA_ERR_SEGMENTS = 4,     /* segment table does not tile the rows                 */
  MLA_ERR_ROWS = 5,         /* protected rows unsorted, duplicated or out of range  */
  MLA_ERR_WORKSPACE = 6,    /* workspace smaller than mla_online_attend_query says  */
  MLA_ERR_HIP = 7           /* a HIP runtime call or kernel launch failed           */
} mla_status;

typedef enum mla_dtype { MLA_BF16 = 0, MLA_F32 = 1 } mla_dtype;

/* Layer geometry (Sec. 2.1, Sec. 3.1).
 *  n_heads        H logical query heads
 *  n_groups       G native output groups; each holds one Global head
 *  d_latent       d_c, width of the latent (the value unless value_rope)
 *  d_rope         d_r, width of the decoupled RoPE key/query part
 *  d_model        width of the projected state z
 *  n_proj_groups  n_pg: the first projection W_a is block-diagonal over n_pg
 *                 projection groups (n_pg = 1 is a dense W_a); n_pg divides G and
 *                 d_model, and d_model/n_pg is a multiple of 32
 *  softmax_scale  factor applied to q.k before the softmax (> 0)
 *  rope_base      RoPE base; frequency j is base^(-2j/d_r), pairs are
 *                 (x_j, x_{j+d_r/2})
 *  value_rope     0: the value is the latent c, a head output has d_v = d_c
 *                 dims and RestorePhase and the inverse output RoPE R^{-1} are
 *                 the identity.  1 (built for (512, 64)): the value is the whole
 *                 latent row [c ; k_r], a head output has d_v = d_c + d_r dims,
 *                 and its RoPE part comes out relative to the query: each
 *                 segment's canonical-frame sum is rotated by R(-(t - p_s)), i.e.
 *                 RestorePhase R(+p_s) then R^{-1} = R(-t) (eq:offonline, Alg. 2).
 *                 Head outputs, partials, the merge and the W_o head blocks are
 *                 then d_v wide.  The attention keeps each head-row's RoPE
 *                 output sums in the workspace (64 KB per work item), which the
 *                 size queries include.                                        */
typedef struct mla_geom {
  int32_t n_heads;
  int32_t n_groups;
  int32_t d_latent;
  int32_t d_rope;
  int32_t d_model;
  int32_t n_proj_groups;
  float softmax_scale;
  double rope_base;
  int32_t value_rope;   /* 0: the value is the d_c latent; 1: the whole latent row
                           (d_c + d_r, its RoPE part rotary) -- see below */
} mla_geom;

/* One document (or the request-query block) of the request (Sec. 2.3; the
 * compact segment-pointer geometry of Sec. 3.2).
 *  kv_start    first storage row of the segment in kv / q_glob / z_off
 *  length      rows in the segment (>= 1)
 *  req_offset  request position of the segment's first row (Delta_i); the
 *              segment's keys are stored in its canonical frame (RoPE at 0..)
 * Across all segments, [kv_start, kv_start+length) tile [0, N) and so do
 * [req_offset, req_offset+length).  Storage row kv_start+u sits at request
 * position req_offset+u.  Segments are identified by their index in the array. */
typedef struct mla_segment {
  int64_t kv_start;
  int64_t length;
  int64_t req_offset;
} mla_segment;

/*
 * Output slots and partials.
 *   Global slot (r, g)    = r*G + g,                  r in [0,N), g in [0,G)
 *   Local slot (a, g, j)  = N*G + (a*G + g)*(hpg-1) + j, for protected row
 *                           prot_rows[a] and the j-th Local head of group g
 *                           (ascending head index, the Global head skipped)
 *   n_slots = N*G + P*G*(hpg-1)
 * A row at request position t sees every segment with req_offset <= t (its own
 * segment causally, keys u <= t - req_offset), in request order.  That list is
 * cut into chunks by `split_keys`:
 *   split_keys == 0  one chunk per visible segment (the per-segment partials of
 *                    SelectiveMLA in Alg. 2);
 *   split_keys  > 0  greedy runs of whole segments in request order; a run is
 *                    closed before a segment that would push its summed segment
 *                    lengths past split_keys (a run holds at least one segment).
 *                    A value >= N gives one chunk per slot: the merge is then
 *                    done entirely inside the attention kernel.
 * Each slot owns one partial per chunk, stored contiguously in request order;
 * part_ptr is the CSR offset array over slots.
 */

/* Size query (host only, pure).  Arguments as for mla_online_attend.  Returns
 * n_slots, n_parts and the workspace bytes mla_online_attend needs. */
mla_status mla_online_attend_query(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                                   const int32_t* prot_rows, int32_t n_prot, int64_t split_keys,
                                   int64_t* n_slots, int64_t* n_parts, size_t* ws_bytes);

/* Steps 1-2: relocation and segment-wise absorbed-MLA attention (Alg. 2,
 * SelectiveMLA with R(-Delta_i) applied to the query; RestorePhase and R^{-1}
 * are the identity when the value is the latent, and are applied to each
 * segment's RoPE output dims when geom->value_rope is set).
 *  geom, segs, n_segs     host; see above
 *  prot_rows, n_prot      host int32 [P], strictly increasing storage rows (the
 *                         protected set A of eq:protected; query rows are
 *                         normally included)
 *  split_keys             >= 0, see above
 *  kv        device bf16 [N, D]: per storage row the latent c (d_c) followed by
 *            the RoPE key in its segment's canonical frame (d_r)
 *  q_glob    device bf16 [N, G, D]: absorbed query of each group's Global head,
 *            RoPE part not yet rotated (it is rotated to the row's position
 *            relative to each segment inside the kernel)
 *  q_loc     device bf16 [P, G, hpg-1, D]: Local-head queries of protected rows
 *            (may be NULL when P == 0 or hpg == 1)
 *  part_o    device f32 [n_parts, d_v]: normalized partial outputs sum p_j v_j / sum p_j
 *  part_lse  device f32 [n_parts]: natural-log log-sum-exp of the scaled scores
 *  part_ptr  device i64 [n_slots + 1]: CSR offsets of each slot's partials
 *  part_seg  device i32 [n_parts, 2] or NULL: first and last segment index
 *            covered by each partial
 *  row_src   device u8 [N] or NULL: 1 where the row is protected (recomputed),
 *            0 where its Local contribution comes from the artifact
 *  workspace device scratch of at least the queried size, 256-byte aligned
 * Errors: NULL, SHAPE, UNSUPPORTED, SEGMENTS, ROWS, WORKSPACE, HIP. */
mla_status mla_online_attend(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                             const int32_t* prot_rows, int32_t n_prot, int64_t split_keys,
                             const void* kv, const void* q_glob, const void* q_loc, float* part_o,
                             float* part_lse, int64_t* part_ptr, int32_t* part_seg, uint8_t* row_src,
                             void* workspace, size_t ws_bytes, void* stream);

/* Step 3: SegmentedLSEMerge (Alg. 2).  For each slot with partials (o_i, l_i):
 * m = max l_i, w_i = exp(l_i - m), O = sum w_i o_i / sum w_i,
 * lse = m + ln sum w_i; a slot with one partial is copied.
 *  n_slots    number of slots (>= 0)
 *  d_latent   head output width d_v: 64, 512, or 576 (512 + 64, rotary value)
 *  part_o, part_lse, part_ptr   device, as written by mla_online_attend
 *                               (part_ptr[0] must be 0, every slot >= 1 partial)
 *  out_dtype  MLA_BF16 or MLA_F32: element type of out_o
 *  out_o      device [n_slots, d_v]; its first N*G rows are O_glob [N, G, d_v]
 *             and the rest O_loc [P, G, hpg-1, d_v]
 *  out_lse    device f32 [n_slots] or NULL
 * Errors: NULL, SHAPE, UNSUPPORTED, HIP. */
mla_status mla_segment_merge(int64_t n_slots, int32_t d_latent, const float* part_o,
                             const float* part_lse, const int64_t* part_ptr, int32_t out_dtype,
                             void* out_o, float* out_lse, void* stream);

/* Step 4: z = W_{a,G} O_G + W_{a,L} O_{L,A} on protected rows, plus z_off on the
 * other rows (eq:offonline, eq:factorization; RestoreAndReplace of Alg. 2).
 * Head h of projection group pg = h / (H/n_pg) uses rows
 * [(h mod H/n_pg)*d_v, +d_v) of w_o[pg] and writes channels
 * [pg*d_model/n_pg, (pg+1)*d_model/n_pg).
 *  geom        host
 *  n_rows      N
 *  o_glob      device bf16 [N, G, d_v]
 *  o_loc       device bf16 [P, G, hpg-1, d_v] (NULL allowed when P == 0 or hpg == 1)
 *  glob_head   host int32 [G]: in-group index (0..hpg-1) of each group's Global head
 *  prot_rows   device int32 [P]: the same strictly increasing protected rows
 *              (read on the device, so not validated; an entry outside [0, N)
 *              is skipped by the Local pass instead of being written)
 *  w_o         device bf16 [n_pg, (H/n_pg)*d_v, d_model/n_pg]
 *  z_off       device bf16 [N, d_model]: projected Local-head artifact; rows in
 *              the protected set are never read (NULL allowed when P == N)
 *  z           device f32 [N, d_model], written
 * Errors: NULL, SHAPE, UNSUPPORTED (also when N x d_model needs more than
 * 2^31 - 8 tiles of 256 rows x 128 channels), ROWS, HIP. */
mla_status mla_sliced_oproj_add(const mla_geom* geom, int64_t n_rows, const void* o_glob,
                                const void* o_loc, const int32_t* glob_head,
                                const int32_t* prot_rows, int32_t n_prot, const void* w_o,
                                const void* z_off, float* z, void* stream);

/* ----------------------------------------------------------------------------
 * Plan once, then attend with the protected set in device memory.
 *
 * In a serving loop the segment table is fixed for a request, while the
 * protected set A is recomputed in every layer on the device (Alg. 2:
 * ProtectedRows, then SelectiveMLA in the same layer; eq:protected).  The
 * calls below split the step accordingly:
 *   mla_online_plan_query  host only: sizes of the plan image and workspace;
 *   mla_online_plan        once per request: builds, on the host, everything
 *                          that depends only on the segment table and uploads it
 *                          into the caller's `plan` buffer (this call stages the
 *                          image through the library's pinned buffer like
 *                          mla_online_attend, so it is not capturable);
 *   mla_online_attend_planned, mla_sliced_oproj_add_planned
 *                          every layer: take prot_rows and |A| from device
 *                          memory, enqueue kernels only (no copy, no memset, no
 *                          host synchronization), and may be captured in a HIP
 *                          graph.  The plan buffer is only read, so any number
 *                          of calls (layers, streams) may share it.
 * prot_cap is the largest |A| the plan accepts; outputs are sized for it.
 * ------------------------------------------------------------------------- */
typedef struct mla_plan_info {
  mla_geom geom;          /* the geometry the plan was built for                          */
  int64_t n_rows;         /* N                                                            */
  int64_t split_keys;     /* chunking, as for mla_online_attend                           */
  int64_t max_slots;      /* N*G + prot_cap*L_h: rows out_o must hold                     */
  int64_t max_parts;      /* largest number of partials of one call (part_seg rows)       */
  int32_t n_segs;
  int32_t prot_cap;       /* largest |A| accepted                                         */
  int32_t max_items;      /* largest number of attention work items of one call           */
  int32_t one_chunk;      /* 1: one chunk per slot, the merge is done inside the attention */
  size_t plan_bytes;      /* device bytes of the plan image                               */
  size_t ws_bytes;        /* device workspace bytes of mla_online_attend_planned          */
  int64_t layout[24];     /* offsets of the plan's and the workspace's tables (library use) */
  uint64_t check;         /* checksum of the fields above, set by the library             */
} mla_plan_info;

/* Sizes only (host, pure): fills *info for the geometry, segment table (as for
 * mla_online_attend), split_keys >= 0 and 0 <= prot_cap <= N.
 * Errors: NULL, SHAPE, UNSUPPORTED, SEGMENTS. */
mla_status mla_online_plan_query(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                                 int64_t split_keys, int32_t prot_cap, mla_plan_info* info);

/* Builds the plan: fills *info as the query does and writes the plan image
 * (info->plan_bytes) into `plan` (device, 256-byte aligned) on `stream`.
 * Errors: as for the query, and WORKSPACE (plan_bytes too small), HIP. */
mla_status mla_online_plan(const mla_geom* geom, const mla_segment* segs, int32_t n_segs, int64_t split_keys,
                           int32_t prot_cap, mla_plan_info* info, void* plan, size_t plan_bytes, void* stream);

/* Steps 1-3 with the protected set in device memory (Alg. 2: SelectiveMLA with
 * the query relocated per segment, and SegmentedLSEMerge): the merged head output
 * and lse of every slot, slot order as for mla_online_attend with the slots of
 * protected row a following prot_rows[a].  With one chunk per slot the merge is
 * the attention kernel's own online rescaling; otherwise the partials live in the
 * workspace and a merge kernel follows in the same call.
 *  geom, info, plan  the geometry (must equal info->geom), and a plan built by
 *                    mla_online_plan (host description and device image)
 *  prot_rows  device int32 [prot_cap]: strictly increasing storage rows; the
 *             first *n_prot are used
 *  n_prot     device int32 [1]: |A|
 *  kv, q_glob as for mla_online_attend; q_loc device bf16 [prot_cap, G, hpg-1, D]
 *             (the first *n_prot rows are read; NULL when hpg == 1)
 *  out_dtype  MLA_BF16 or MLA_F32: element type of out_o
 *  out_o      device [info->max_slots, d_v]: rows [0, N*G + |A|*L_h) written
 *  out_lse    device f32 [info->max_slots] or NULL: natural-log lse of each slot
 *  part_ptr   device i64 [info->max_slots + 1] or NULL: CSR offsets of each slot's
 *             partials (entries [0, n_slots] written)
 *  part_seg   device i32 [info->max_parts, 2] or NULL (needs part_ptr): first and
 *             last segment of each partial
 *  row_src    device u8 [N] or NULL: 1 on protected rows
 *  status     device int32 [1] or NULL: MLA_OK, or MLA_ERR_ROWS when the device
 *             list was rejected (|A| > prot_cap or < 0, a row outside [0, N), not
 *             strictly increasing); the call then writes no output row
 *             (MLA_ERR_WORKSPACE would mean the plan's bounds were exceeded,
 *             which they cannot be for a list of at most prot_cap rows)
 *  workspace  device, 256-byte aligned, info->ws_bytes; overwritten
 * Host errors (nothing enqueued): NULL, SHAPE (also a geometry or info that does
 * not match), WORKSPACE, HIP. */
mla_status mla_online_attend_planned(const mla_geom* geom, const mla_plan_info* info, const void* plan,
                                     const int32_t* prot_rows, const int32_t* n_prot, const void* kv,
                                     const void* q_glob, const void* q_loc, int32_t out_dtype, void* out_o,
                                     float* out_lse, int64_t* part_ptr, int32_t* part_seg, uint8_t* row_src,
                                     int32_t* status, void* workspace, size_t ws_bytes, void* stream);

/* For callers that cannot allocate (code under HIP graph capture that must not
 * create memory, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation as mla_online_attend_planned with the workspace replaced by a
 * library-owned device array of MLA_NOALLOC_SCRATCH_BYTES per GPU (allocated
 * with the library's code on each GPU and held until the process ends).  The
 * call allocates nothing: it validates on the host, looks the array's address
 * up once per device (hipGetSymbolAddress) and enqueues kernels.
 *  Arguments as for mla_online_attend_planned, without workspace / ws_bytes.
 *  A plan whose workspace needs more than MLA_NOALLOC_SCRATCH_BYTES (a chunked
 *  plan's partials, a very large work list, or a rotary-value plan's
 *  accumulators beyond a few hundred work items) returns MLA_ERR_WORKSPACE
 *  before anything is enqueued; one-chunk plans of the 256K workload with the
 *  latent value need about 4 MB.
 *  Every call on a GPU uses that GPU's one array, which keeps the last call's
 *  contents (each call writes every entry before reading it): calls that
 *  overlap on one GPU (two streams, two host threads) race and must be
 *  serialized by the caller. */
#define MLA_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
mla_status mla_online_attend_planned_noalloc(const mla_geom* geom, const mla_plan_info* info, const void* plan,
                                             const int32_t* prot_rows, const int32_t* n_prot, const void* kv,
                                             const void* q_glob, const void* q_loc, int32_t out_dtype, void* out_o,
                                             float* out_lse, int64_t* part_ptr, int32_t* part_seg,
                                             uint8_t* row_src, int32_t* status, void* stream);

/* Step 4 with the protected set in device memory: as mla_sliced_oproj_add, with
 * |A| read from the device (clamped to [0, info->prot_cap]) and z in f32 or bf16.
 *  o_glob, o_loc  the first N*G rows of out_o and the rows after them
 *  prot_rows, n_prot  as for mla_online_attend_planned (entries outside [0, N)
 *             are skipped by the Local pass, as in mla_sliced_oproj_add)
 *  z_dtype    MLA_F32 or MLA_BF16 (the latter is what mla_shared_wb takes; a
 *             protected row then carries the rounding of its Local sum and of z)
 * Errors: NULL, SHAPE, UNSUPPORTED, HIP. */
mla_status mla_sliced_oproj_add_planned(const mla_geom* geom, const mla_plan_info* info, const void* o_glob,
                                        const void* o_loc, const int32_t* glob_head, const int32_t* prot_rows,
                                        const int32_t* n_prot, const void* w_o, const void* z_off, int32_t z_dtype,
                                        void* z, void* stream);

/* ----------------------------------------------------------------------------
 * mla_offline_produce -- the MLA-Off native producer (Alg. 1, NativeProducer;
 * eq:offonline): the Local-head artifact of every row of every segment,
 *   z_off[r] = sum_{h Local} W_block(h)^T O_h^can[r],
 * where O_h^can[r] attends only to the keys of r's own segment with canonical
 * offsets u' <= u_r, the query's RoPE part rotated to its canonical position
 * u_r (the segment evaluated alone, its first row at position 0).  The result is
 * what mla_sliced_oproj_add reads as z_off.  Every segment of the table is
 * produced, the query block included (a caller that only needs document rows
 * ignores the others).
 *
 *   geom           as for mla_sliced_oproj_add (n_proj_groups, d_model used).
 *   segs, n_segs   segment table as for mla_online_attend (host).
 *   kv             [N, D] bf16 device: packed latent || canonical RoPE key.
 *   q_loc          [N, G, hpg-1, D] bf16 device: the Local-head queries of every
 *                  row (Local heads of group g in ascending head index, the
 *                  Global head glob_head[g] skipped); RoPE part unrotated.
 *   glob_head      [G] host: in-group index of each group's Global head.
 *   w_o            as for mla_sliced_oproj_add.
 *   out_dtype      MLA_BF16 or MLA_F32: element type of z_off.
 *   z_off          [N, d_model] device, written (every element).
 *   workspace      device, 256-byte aligned, at least the size returned by
 *                  mla_offline_produce_query: plan (with a rotary value its
 *                  accumulators), bf16 head outputs [N, G, hpg-1, d_v].
 *                  Overwritten.
 * With hpg == 1 (no Local heads) z_off is written with zeros.  Errors as for
 * mla_online_attend.
 * ------------------------------------------------------------------------- */
mla_status mla_offline_produce_query(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                                     size_t* ws_bytes);

mla_status mla_offline_produce(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                               const void* kv, const void* q_loc, const int32_t* glob_head,
                               const void* w_o, int32_t out_dtype, void* z_off, void* workspace,
                               size_t ws_bytes, void* stream);

/* ----------------------------------------------------------------------------
 * mla_protected_rows -- the protected token-row set of Sec. 2.3 (eq:protected):
 *   A = Q u N u D u B_edge u I_top u T_tail
 * as an ascending list of storage rows, ready to be copied to the host as the
 * prot_rows argument of mla_online_attend.
 *   Q       rows of the query segment (cfg->query_seg, -1 for none);
 *   N, D    rows flagged new (bit 0 of row_flags) or dirty (bit 1);
 *   B_edge  the first and last cfg->edge_rows rows of every relocated segment,
 *           i.e. every non-query segment whose request offset is not 0;
 *   T_tail  rows whose true request position is among the last cfg->tail_rows;
 *   I_top   the highest-scoring candidate rows outside the sets above, where
 *           candidates are the rows that have an artifact (neither query nor
 *           new rows): enough of them that round(cfg->budget * |candidates|)
 *           candidates are protected (none when the other sets already reach
 *           it); the budget is the controller's level (0.10, 0.20 or 0.25 in the
 *           paper).  Scores rank by IEEE-754 totalOrder, descending; equal
 *           scores go to the lower row; rounding is half up.
 *
 *   segs, n_segs   segment table as for mla_online_attend (host).
 *   cfg            host; edge_rows >= 0, tail_rows >= 0, 0 <= budget <= 1.
 *   row_flags      [N] uint8 device, or NULL (no new or dirty rows).
 *   index_scores   [N] float device (the Indexer's score of each row), or NULL
 *                  (every score equal: I_top then takes the lowest rows).
 *   prot_rows      [N] int32 device, written with the |A| protected rows.
 *   n_prot         [1] int32 device, written with |A|.
 *   workspace      device, 256-byte aligned, mla_protected_rows_query bytes.
 * Errors as for mla_online_attend; the result is exact (integer), independent
 * of the launch configuration.
 * ------------------------------------------------------------------------- */
typedef struct mla_protect_cfg {
  int32_t query_seg;   /* index of the query segment in segs, or -1                 */
  int32_t edge_rows;   /* B: first / last rows of each relocated segment (128)      */
  int64_t tail_rows;   /* T: most recent rows in request order (32768)              */
  double budget;       /* protected share of candidate rows (0.10, 0.20, 0.25)      */
} mla_protect_cfg;

mla_status mla_protected_rows_query(const mla_segment* segs, int32_t n_segs, size_t* ws_bytes);

mla_status mla_protected_rows(const mla_segment* segs, int32_t n_segs, const mla_protect_cfg* cfg,
                              const uint8_t* row_flags, const float* index_scores,
                              int32_t* prot_rows, int32_t* n_prot, void* workspace, size_t ws_bytes,
                              void* stream);

/* The protected set on the plan-once path: the same set as mla_protected_rows,
 * with the segment table read from a plan built by mla_online_plan (it holds
 * the storage-ordered table), so the call only enqueues kernels (its control
 * words are cleared by a kernel, not uploaded) and may be captured in a HIP
 * graph together with mla_online_attend_planned, which takes its prot_rows and
 * n_prot directly (Alg. 2: ProtectedRows, then SelectiveMLA in the same layer).
 *  info, plan     a plan from mla_online_plan (host description, device image);
 *                 query_seg indexes the plan's segment table
 *  cfg, row_flags, index_scores, prot_rows [N], n_prot   as for mla_protected_rows
 *  workspace      device, 256-byte aligned, mla_protected_rows_planned_query bytes
 *                 (17 B per row plus 16.6 KB)
 * Errors: NULL, SHAPE (also an info not written by mla_online_plan), WORKSPACE, HIP. */
mla_status mla_protected_rows_planned_query(const mla_plan_info* info, size_t* ws_bytes);

mla_status mla_protected_rows_planned(const mla_plan_info* info, const void* plan, const mla_protect_cfg* cfg,
                                      const uint8_t* row_flags, const float* index_scores, int32_t* prot_rows,
                                      int32_t* n_prot, void* workspace, size_t ws_bytes, void* stream);

/* ----------------------------------------------------------------------------
 * mla_moe_fanout -- the adaptive MoE fanout of Sec. 2.4 (eq:moe) for the
 * reusable middle layers.  For every token row the router's top_k experts are
 * ranked by weight (IEEE-754 totalOrder, descending; equal weights go to the
 * lower expert index), and the fanout is
 *   K = min{k in [min_k, top_k] : sum_{j<=k} p_(j) / sum_{r<=top_k} p_(r) >= tau}
 * (top_k when no k qualifies, e.g. when the top_k weights sum to 0).  The paper
 * uses top_k = 6 and min_k = 3; fence layers keep all six (tau > 1).  The
 * executed experts are the first K of the ranked list and keep their original
 * weights: the normalization only decides K.  K is decided in float32: the sum
 * of the top_k weights left to right, each share a correctly rounded division,
 * the shares accumulated left to right and compared with tau.
 *
 *   n_rows, n_experts  N token rows, E routed experts (top_k <= E <= 1024).
 *   router        [N, E] float device: the router's weights p.
 *   top_k, min_k  1 <= min_k <= top_k <= 8.
 *   tau           the fanout threshold (any non-NaN value).
 *   expert_idx    [N, top_k] int32 device, written: experts by rank.
 *   expert_w      [N, top_k] float device, written: their weights p.
 *   fanout        [N] int32 device, written: K.
 *   expert_count  [E] int32 device or NULL: written with the number of rows
 *                 that execute each expert (rank < K).
 * All device arrays 4-byte aligned.  Errors as for mla_online_attend; the
 * outputs are exact (integer ranks and copies of the inputs).
 * ------------------------------------------------------------------------- */
mla_status mla_moe_fanout(int64_t n_rows, int32_t n_experts, const float* router, int32_t top_k, int32_t min_k,
                          float tau, int32_t* expert_idx, float* expert_w, int32_t* fanout,
                          int32_t* expert_count, void* stream);

/* ----------------------------------------------------------------------------
 * mla_shared_wb -- the shared second output projection y = W_b z that every row's
 * group-sliced state z meets after the artifact add (Sec. 2.1 eq:factorization,
 * Alg. 2 returns W_b z).  bf16 MFMA with fp32 accumulation.
 *
 *   n_rows, d_in, d_out  N rows; z width (a multiple of 64, at most 16384);
 *                  output channels (>= 1).
 *   z              [N, d_in] bf16 device (the state z, in bf16).
 *   w_b            [d_out, d_in] bf16 device (a linear layer's weight: row o holds
 *                  the d_in weights of output channel o).
 *   out_dtype      MLA_BF16 or MLA_F32 for y.
 *   y              [N, d_out] device, written.
 * Device arrays 16-byte aligned.  Errors as for mla_online_attend.
 * ------------------------------------------------------------------------- */
mla_status mla_shared_wb(int64_t n_rows, int32_t d_in, int32_t d_out, const void* z, const void* w_b,
                         int32_t out_dtype, void* y, void* stream);

/* Static description of a status code. */
const char* mla_status_str(mla_status s);

/* Detail of the calling thread's last failed call ("" if none). */
const char* mla_last_error_detail(void);

/* Library version string. */
const char* mla_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MLA_ONLINE_H */
