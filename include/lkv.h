/*
 * lkv.h -- C ABI of liblkv.so, the gfx950 (MI355X) implementation of one
 * recurrent layer's online prefill in LinearKV's hybrid position-independent
 * caching: initialise the layer's state from K cached per-block states, then
 * run the chunkwise recurrence over the request's online tokens.
 *
 * Notation.  For one value head the state is S in R^{dv x dk}, row-major
 * (dk contiguous).  The paper writes the state as its transpose, S_paper in
 * R^{dk x dv} with S_i = T_i S_{i-1} + u_i (Sec. 2, Eq. 1); here the same
 * recurrence is S_t = S_{t-1} A_t + (update), with
 *   Gated DeltaNet (Eq. 3): A_t = alpha_t (I - beta_t k_t k_t^T),
 *       alpha_t = exp(g_t), update beta_t v_t k_t^T, output o_t = scale * S_t q_t;
 *   Mamba-2 (Eq. 2): A_t = exp(dt_t A_h) I, update dt_t x_t B_t^T,
 *       output y_t = S_t C_t.
 * A block of tokens maps any incoming state to S_out = S_in M + B (Eq. 5):
 * B is the state it reaches from zero, M = A_1 ... A_L its transition (a dense
 * dk x dk matrix for Gated DeltaNet, the scalar exp(Lambda), Lambda =
 * A_h sum dt, for Mamba-2).
 *
 * Memory.  Every pointer argument that names tensor data is a DEVICE pointer
 * owned by the caller; the library never allocates, frees or synchronises.
 * Tensors are dense, row-major, and 16-byte aligned.  Token streams are packed
 * "THD": [n_tok, heads, dim] over consecutive segments, cu[s]..cu[s+1] being
 * segment s's tokens.  Value head h reads q/k head h / (h_v / h_qk).
 *
 * Calls.  Every call validates its arguments on the host, enqueues its kernels
 * on `stream` (a hipStream_t; NULL = the null stream) and returns without
 * waiting.  Outputs are fully overwritten.  Results are deterministic: the
 * same inputs give bitwise-identical outputs run to run.  Argument errors are
 * reported synchronously through the return code; a failed launch returns
 * LKV_E_HIP and lkv_last_hip_error() gives the HIP code.  Device-side index
 * checks never fault: segment offsets are clamped to [0, n_tok], and a block
 * index outside [0, n_blk) turns that request's whole output slice into NaN.
 * Calls that overlap on one stream are ordered by the stream; calls on
 * different streams that share an output race.
 */
#ifndef LKV_H
#define LKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LKV_ABI_VERSION 9

typedef enum {
    LKV_OK = 0,
    LKV_E_NULL = 1,         /* a required pointer is NULL                         */
    LKV_E_SHAPE = 2,        /* a size is negative, zero where it may not be, or inconsistent */
    LKV_E_DTYPE = 3,        /* unknown or unsupported dtype for this argument        */
    LKV_E_ALIGN = 4,        /* a tensor pointer is not 16-byte aligned               */
    LKV_E_UNSUPPORTED = 5,  /* a valid geometry this build does not implement        */
    LKV_E_WORKSPACE = 6,    /* beyond the allocation-free variant's fixed scratch     */
    LKV_E_HIP = 7           /* the HIP runtime reported an error (lkv_last_hip_error) */
} lkv_status;

typedef enum { LKV_F32 = 0, LKV_BF16 = 1 } lkv_dtype;
typedef enum { LKV_GDN = 0, LKV_SSD = 1 } lkv_family;

/* Geometry of one recurrent layer.
 *   family     LKV_GDN | LKV_SSD
 *   h_qk       GDN: q/k heads        | SSD: B/C groups G           (h_v % h_qk == 0)
 *   h_v        GDN: value heads      | SSD: heads H                (one state each)
 *   dk         GDN: key dim          | SSD: state dim N            in {16, 32, 64, 128}
 *   dv         GDN: value dim        | SSD: head dim P             multiple of 16, <= 512
 *   chunk      tokens per chunk of the chunkwise kernels           in {16, 64}
 *   io_dtype   dtype of q/k/v (C/B/x) and o (y)                    LKV_F32 | LKV_BF16
 *              (LKV_F32 requires dk <= 64)
 *   gate_dtype GDN: dtype of g = log(alpha) and beta               LKV_F32 | LKV_BF16
 *              SSD: must be LKV_F32 (dt)                                              */
typedef struct {
    int32_t family;
    int32_t h_qk;
    int32_t h_v;
    int32_t dk;
    int32_t dv;
    int32_t chunk;
    int32_t io_dtype;
    int32_t gate_dtype;
} lkv_layer;

/* One packed token stream over n_seq segments (cached blocks or requests).
 *   cu       device int32 [n_seq+1], cu[0] = 0, non-decreasing, cu[n_seq] = n_tok
 *   n_seq    number of segments (>= 0)
 *   n_tok    host copy of cu[n_seq]
 *   q        GDN q [n_tok,h_qk,dk] | SSD C [n_tok,G,N]   (unused by lkv_block_summary)
 *   k        GDN k [n_tok,h_qk,dk] | SSD B [n_tok,G,N]
 *   v        GDN v [n_tok,h_v,dv]  | SSD x [n_tok,H,P]
 *   g        GDN g = log(alpha) [n_tok,h_v] (gate_dtype) | SSD dt [n_tok,H] f32, > 0
 *   beta     GDN beta [n_tok,h_v] (gate_dtype)           | SSD unused (NULL)
 *   A        GDN unused (NULL)                           | SSD A [H] f32, < 0          */
typedef struct {
    const int32_t* cu;
    int32_t n_seq;
    int64_t n_tok;
    const void* q;
    const void* k;
    const void* v;
    const void* g;
    const void* beta;
    const float* A;
} lkv_tokens;

/* ABI version of the loaded library (LKV_ABI_VERSION). */
int lkv_abi_version(void);

/* Static English text for a status code. */
const char* lkv_status_string(lkv_status s);

/* hipError_t behind the last LKV_E_HIP returned on the calling thread. */
int lkv_last_hip_error(void);

/* Bound of the chunk kernels' one inter-wave wait.  Within a workgroup of the
 * Gated DeltaNet chunk kernels (lkv_block_summary, lkv_gdn_chunk_scan,
 * lkv_chunk_scan_from_pool), one wave inverts the diagonal blocks of
 * (I + diag(beta) strictly-lower(K K^T)) -- the delta rule's triangular system
 * of the chunkwise form of Eq. 3 -- after the waves that mask them signal
 * through a counter in LDS.  That wait polls the counter at most `polls` times
 * (with a short sleep between polls).  A wait that gives up stores NaN blocks,
 * so the chunk's state rows and outputs, and every later chunk's, become NaN:
 * a missed signal is visible in the results, never silently wrong, and every
 * kernel still ends.  The default, 16384 polls, is about a millisecond, against
 * well under 200 polls for a legitimate wait; 0 never polls, so every wait
 * gives up (a host-forced failure for tests); a negative value restores the
 * default.  Process-wide; read by each call when it launches.  Returns the
 * previous bound. */
int32_t lkv_set_wait_limit(int32_t polls);

/* Per-block summary (Eq. 5): for every segment of `blocks`, scanned from an
 * empty start, write
 *   B_out  [n_blk,h_v,dv,dk] f32   the block's final state from zero (S_local)
 *   M_out  GDN: [n_blk,h_v,dk,dk] f32, M = A_1...A_L, row-major M[i][j]
 *          SSD: [n_blk,H] f32, the log-decay Lambda = A_h * sum_t dt_t
 * Either output may be NULL (then it is not computed); not both.
 * blocks->q is not read; with B_out NULL neither is blocks->v (it may be
 * NULL), and for Mamba-2 only dt and A are read (k may be NULL too).  Errors: LKV_E_NULL, LKV_E_SHAPE, LKV_E_DTYPE,
 * LKV_E_ALIGN, LKV_E_UNSUPPORTED, LKV_E_HIP. */
lkv_status lkv_block_summary(const lkv_layer* layer, const lkv_tokens* blocks,
                             float* B_out, float* M_out, void* stream);

/* Single-block initialisation (Sec. 3.2, "single-block initialization"):
 *   S_init[r] = B_pool[src_blk[r]]   (bit-exact copy), for r < n_req.
 *   B_pool   [n_blk,h_v,dv,dk] f32 device
 *   src_blk  device int32 [n_req]; -1 gives a zero state; any other value
 *            outside [0, n_blk) gives a NaN slice
 *   S_init   [n_req,h_v,dv,dk] f32 device; must not overlap B_pool
 * The paper's default picks each request's last matched block; any choice
 * (e.g. a random block, its App. A variant) is the caller's. */
lkv_status lkv_init_single(const lkv_layer* layer, int32_t n_req, int32_t n_blk,
                           const float* B_pool, const int32_t* src_blk, float* S_init,
                           void* stream);

/* Exact composition (Eq. 6, evaluated as Eq. 5 applied block after block from
 * an empty prefix): for request r with blocks b_1..b_K (context order)
 *   S <- B_{b_1};  S <- S M_{b_j} + B_{b_j} for j = 2..K;  S_init[r] = S
 * (Mamba-2: S <- exp(Lambda_{b_j}) S + B_{b_j}).  K = 0 gives zeros.
 *   B_pool   [n_blk,h_v,dv,dk] f32 device
 *   M_pool   GDN [n_blk,h_v,dk,dk] f32 (row-major M) | SSD [n_blk,H] f32 Lambda.
 *            The entry of each request's first block is never read.
 *   blk_ids  device int32 [n_ids]: every request's pool rows, concatenated
 *   blk_cu   device int32 [n_req+1]: request r uses blk_ids[blk_cu[r]..blk_cu[r+1]),
 *            clamped to [0, n_ids]; an id outside [0, n_blk) gives a NaN slice
 *   n_ids    host copy of blk_cu[n_req]
 *   S_init   [n_req,h_v,dv,dk] f32 device; must not overlap the pools          */
lkv_status lkv_init_compose(const lkv_layer* layer, int32_t n_req, int32_t n_blk,
                            const float* B_pool, const float* M_pool,
                            const int32_t* blk_ids, const int32_t* blk_cu, int32_t n_ids,
                            float* S_init, void* stream);

/* Gated DeltaNet chunkwise scan over each request's online tokens (Alg. 1,
 * recompute step; Eq. 1 and Eq. 3), starting from S_init:
 *   o[t]     = scale * S_t q_t, stored in io_dtype, [n_tok,h_v,dv]
 *   S_final  [n_req,h_v,dv,dk] f32, the state after the last token
 * S_init may be NULL (zero start) and may equal S_final (in place).
 * o may be NULL (state only).  layer->family must be LKV_GDN. */
lkv_status lkv_gdn_chunk_scan(const lkv_layer* layer, const lkv_tokens* online, float scale,
                              const float* S_init, void* o, float* S_final, void* stream);

/* Mamba-2 (SSD) chunkwise scan (Eq. 1 and Eq. 2): y[t] = S_t C_t in io_dtype
 * [n_tok,H,P]; S_final [n_req,H,P,N] f32.  S_init may be NULL or equal
 * S_final; y may be NULL.  layer->family must be LKV_SSD. */
lkv_status lkv_ssd_chunk_scan(const lkv_layer* layer, const lkv_tokens* online,
                              const float* S_init, void* y, float* S_final, void* stream);

/* LinearKV's path in one launch: the chunk scan of lkv_gdn_chunk_scan /
 * lkv_ssd_chunk_scan (by layer->family) whose initial state for request r is
 * the cached state B_pool[src_blk[r]] itself, read by the scan kernel (Sec.
 * 3.2, single-block initialisation; App. A for other choices of the block).
 * The results are bit-identical to lkv_init_single (or lkv_init_single_bf16)
 * followed by the scan from its output, without the intermediate state buffer.
 *   B_pool     [n_blk,h_v,dv,dk] device, pool_dtype LKV_F32 or LKV_BF16 (widened
 *              exactly); may be NULL when n_blk = 0
 *   src_blk    device int32 [online->n_seq]: -1 gives a zero start, any other
 *              value outside [0, n_blk) a NaN state
 *   scale      Gated DeltaNet output scale (ignored for Mamba-2)
 *   out, S_final as for the scans.
 * Errors: as for the scans, plus LKV_E_DTYPE for an unknown pool_dtype. */
lkv_status lkv_chunk_scan_from_pool(const lkv_layer* layer, const lkv_tokens* online, float scale,
                                    const void* B_pool, int32_t pool_dtype, int32_t n_blk,
                                    const int32_t* src_blk, void* out, float* S_final, void* stream);

/* Sequence-parallel chunk scan.  The results of lkv_gdn_chunk_scan /
 * lkv_ssd_chunk_scan (by layer->family; `scale` is ignored for Mamba-2),
 * computed with the sequence dimension split: each request's online stream
 * is cut into `pieces` consecutive pieces of whole chunks (the last takes the
 * remainder; trailing pieces may be empty), and the recurrence is Eq. 5
 * applied piece after piece.  Every piece's pair (its end state from zero and
 * its transition -- the dense M of Gated DeltaNet, the log-decay of Mamba-2)
 * is computed at once, as by lkv_block_summary; composing the request's
 * initial state with the pairs of pieces 0..p-1 (Eq. 6 from a non-empty
 * prefix, as lkv_init_compose) gives piece p's start state and, after the last
 * piece, the final state; then every piece is scanned from its start state,
 * all at once, for the outputs.  The chain of dependent chunks per request is
 * about pieces times shorter, at the price of the pieces' transitions
 * (Gated DeltaNet: about twice the state work of a scan without outputs;
 * Mamba-2: a sum of dt) and the composition: it pays when few (request, head)
 * chains leave the GPU idle, e.g. one 8K request.  Results agree with the
 * serial scan within the fp32 state tolerance (they are not bit-identical:
 * the rounding order differs).
 *   pieces   1..64
 *   ws       device workspace of at least lkv_chunk_scan_sp_workspace bytes,
 *            256-byte aligned, caller-owned; its contents on entry do not
 *            matter and are overwritten.  Calls that share a workspace race
 *            unless ordered by a stream.
 * Other arguments as in lkv_gdn_chunk_scan (S_init may be NULL: zero start;
 * S_final may be NULL, but S_init must not alias S_final here).  Errors:
 * LKV_E_NULL, LKV_E_SHAPE (also a workspace too small), LKV_E_DTYPE,
 * LKV_E_ALIGN, LKV_E_UNSUPPORTED, LKV_E_HIP. */
lkv_status lkv_chunk_scan_sp_workspace(const lkv_layer* layer, int32_t n_req, int32_t pieces,
                                       size_t* bytes);
lkv_status lkv_chunk_scan_sp(const lkv_layer* layer, const lkv_tokens* online, float scale,
                             const float* S_init, void* out, float* S_final, int32_t pieces,
                             void* ws, size_t ws_bytes, void* stream);

/* Allocation-free variant of lkv_chunk_scan_sp, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and results, bit for
 * bit, with the workspace taken from a fixed scratch array of 64 MiB that the
 * library's device code holds on every GPU it runs on until the process ends.
 * The call allocates and frees nothing.  Arguments as in lkv_chunk_scan_sp,
 * without the workspace; a call whose workspace (lkv_chunk_scan_sp_workspace)
 * exceeds 64 MiB returns LKV_E_WORKSPACE and launches nothing (at dk = dv =
 * 128 and 32 heads a state takes 2 MiB, so e.g. one request in up to 6
 * pieces fits, Mamba-2 with 64 heads of 64 x 128 one request in up to 15).
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (on different streams, or from several threads) race and must be ordered
 * by the caller.  No part of the array needs clearing between calls (every
 * byte a call reads it has first written).  The first call on a device, with
 * that device current, looks up the array's device address (no allocation).
 * Errors: as lkv_chunk_scan_sp, and LKV_E_WORKSPACE. */
lkv_status lkv_chunk_scan_sp_noalloc(const lkv_layer* layer, const lkv_tokens* online, float scale,
                                     const float* S_init, void* out, float* S_final, int32_t pieces,
                                     void* stream);

/* Decode step: the step that follows the online prefill, which keeps only the
 * final state for it (Sec. 2).  One new token per request advances each
 * request's state by one step of the recurrence (Eq. 1) and gives that
 * token's output, with the post-update state:
 *   Gated DeltaNet (Eq. 3): S <- alpha S + beta (v - alpha S k) k^T
 *                           (= S A_t + beta v k^T),  o = scale * S q
 *   Mamba-2 (Eq. 2):        S <- exp(dt A_h) S + dt x B^T,  y = S C
 *   q, k   [n_req,h_qk,dk] io_dtype          (SSD: C, B)
 *   v      [n_req,h_v,dv]  io_dtype          (SSD: x)
 *   g, beta GDN: [n_req,h_v] gate_dtype, g = log(alpha)
 *   dt, A  SSD: dt [n_req,H] f32 (> 0), A [H] f32 (< 0)
 *   S      [n_req,h_v,dv,dk] f32 device, read and updated in place
 *   o / y  [n_req,h_v,dv] io_dtype, or NULL (state only)
 * q, k, v and S must be 16-byte aligned.  layer->chunk is not used.  The call
 * is memory-bound: it reads and writes every state element once.
 * Errors: LKV_E_NULL, LKV_E_SHAPE, LKV_E_DTYPE, LKV_E_ALIGN, LKV_E_UNSUPPORTED,
 * LKV_E_HIP. */
lkv_status lkv_gdn_decode(const lkv_layer* layer, int32_t n_req, const void* q, const void* k,
                          const void* v, const void* g, const void* beta, float scale, float* S,
                          void* o, void* stream);
lkv_status lkv_ssd_decode(const lkv_layer* layer, int32_t n_req, const void* C, const void* B,
                          const void* x, const float* dt, const float* A, float* S, void* y,
                          void* stream);

/* bf16 cached-state pool.  The cache stores each block's end state S_local in
 * bf16 in host memory and loads it at serving time (Sec. 4, environment).
 * These variants of the two initialisations read B_pool as bf16
 * [n_blk,h_v,dv,dk] and widen it exactly to fp32 (bf16 -> fp32 appends zero
 * mantissa bits); everything else, M_pool included (it comes from the online
 * fold, in fp32), is as in lkv_init_single / lkv_init_compose.  In particular
 * lkv_init_single_bf16 is a bit-exact widening copy. */
lkv_status lkv_init_single_bf16(const lkv_layer* layer, int32_t n_req, int32_t n_blk,
                                const void* B_pool, const int32_t* src_blk, float* S_init,
                                void* stream);
lkv_status lkv_init_compose_bf16(const lkv_layer* layer, int32_t n_req, int32_t n_blk,
                                 const void* B_pool, const float* M_pool,
                                 const int32_t* blk_ids, const int32_t* blk_cu, int32_t n_ids,
                                 float* S_init, void* stream);

/* Round n fp32 values (device) to bf16 (device), round to nearest even; NaN
 * stays NaN (quiet), infinities and signed zeros are kept, values beyond the
 * bf16 range round to infinity.  This is the storage step of a computed pool
 * (e.g. lkv_block_summary's B_out) into the cache's bf16 format.  src and dst
 * 16-byte aligned, not overlapping.  Errors: LKV_E_NULL, LKV_E_SHAPE,
 * LKV_E_ALIGN, LKV_E_HIP. */
lkv_status lkv_round_bf16(const float* src, void* dst, int64_t n, void* stream);

/* Host-to-device staging of cache rows (the serving-time load of the cached
 * artefacts from host memory, Sec. 4; the transfer the paper leaves as future
 * work, Sec. 4.3): for i < n_rows, dst row i <- src row rows[i], rows being
 * row_bytes bytes.  src is HOST memory and should be pinned (hipHostMalloc):
 * then the copies are asynchronous on `stream` and overlap kernels running
 * on other streams; from pageable memory they are synchronous.  rows is a
 * HOST int32 array (>= 0, not bounds-checked against src: the caller owns
 * src's extent); each run of consecutive rows is one copy.  dst is device
 * memory of n_rows * row_bytes bytes.  Typical use: a batch's single-block
 * rows (one per request) or its exact-composition rows (K per request),
 * staged into a compact device pool indexed by the remapped row numbers.
 * Errors: LKV_E_NULL, LKV_E_SHAPE, LKV_E_HIP. */
lkv_status lkv_stage_rows(void* dst, const void* src, const int32_t* rows, int32_t n_rows,
                          int64_t row_bytes, void* stream);

/* Selected-position gather (Alg. 1, selection and recompute steps): the
 * recompute runs the recurrence over the selected positions U = {i_1 < ... <
 * i_m} of each request's context only, in context order (Sec. 3.1), so its
 * token stream is the context's rows at U.  For request r and every selected
 * row j in [sel_cu[r], sel_cu[r+1]):
 *   out row j  =  context row ctx->cu[r] + pos[j]   (bit-exact, each array)
 *   ctx      the requests' full context streams (n_seq = n_req)
 *   pos      device int32 [n_sel], positions inside the request's context.
 *            Context order is the caller's: the call copies in the given
 *            order and does not sort or check it.  A position outside
 *            [0, context length) gives NaN rows.
 *   sel_cu   device int32 [n_req+1] (clamped to [0, n_sel]); rows outside
 *            every segment get NaN rows
 *   n_sel    host copy of sel_cu[n_req]
 *   q, k, v, g, beta  outputs [n_sel, ...] in ctx's dtypes and row shapes;
 *            each may be NULL (not gathered), and then ctx's may be NULL too.
 *            SSD: q = C, k = B, v = x, g = dt, beta unused.
 * The outputs with ctx->A form the online stream of the chunk scan, with
 * cu = sel_cu.  Outputs must not overlap ctx.  HBM-bound: every gathered byte
 * is read once and written once.  Errors: LKV_E_NULL, LKV_E_SHAPE,
 * LKV_E_DTYPE, LKV_E_ALIGN, LKV_E_UNSUPPORTED, LKV_E_HIP. */
lkv_status lkv_gather_selected(const lkv_layer* layer, const lkv_tokens* ctx, const int32_t* pos,
                               const int32_t* sel_cu, int64_t n_sel, void* q, void* k, void* v,
                               void* g, void* beta, void* stream);

/* Relative-error diagnostic (Sec. 3.2, the probe of the constructed initial
 * state against the true full-prefix state S*, before any recomputation):
 * for slice s < n_slices (slice_elems consecutive fp32 values of S and S_ref,
 * e.g. one (request, head) state),
 *   sq[2s] = ||S_s - R_s||_F^2,   sq[2s+1] = ||R_s||_F^2     (fp64 sums)
 *   rel[s] = sqrt(sq[2s]) / sqrt(sq[2s+1])
 * and, when rel_group is not NULL, for g < n_slices / group over the slices
 * g*group .. g*group+group-1 (e.g. all heads of one request's layer, the
 * paper's per-layer figure)
 *   rel_group[g] = sqrt(sum sq[2s]) / sqrt(sum sq[2s+1]).
 * IEEE division: a zero reference gives inf, or NaN when S is zero too.
 * Inputs are device fp32, 16-byte aligned, slice_elems a multiple of 4;
 * outputs are device fp64 (sq [2*n_slices], rel [n_slices], rel_group
 * [n_slices/group]).  group must divide n_slices.  With the composed error
 * e = S - S* the squared norms follow the mismatch recursion of Eq. 7 for
 * perturbed summaries.  Errors: LKV_E_NULL, LKV_E_SHAPE, LKV_E_ALIGN, LKV_E_HIP. */
lkv_status lkv_state_rel_error(const float* S, const float* S_ref, int32_t n_slices,
                               int64_t slice_elems, int32_t group, double* sq, double* rel,
                               double* rel_group, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LKV_H */
