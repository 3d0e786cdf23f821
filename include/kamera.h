/*
 * kamera.h -- C ABI of the Kamera chunk-reuse operator for AMD Instinct MI355X
 * (gfx950).
 *
 * Kamera (arxiv 2606.23581) stores each cached chunk position-free -- the
 * pre-RoPE keys and the values of every layer and KV head, or an MLA latent
 * plus its decoupled rope key -- together with a rank-m "conditioning patch"
 * per layer and head (Eq. eq:operator, Sec. 1; Sec. 3).  Reusing the chunk at
 * a new position needs no forward pass: the keys are re-rotated to the target
 * position and the patch is added back (App. A, serve step).  This library
 * performs that serve step on the GPU:
 *
 *   kamera_rehydrate     K' = R(pos) (K + U_k W_k),  V' = V + U_v W_v,
 *                        into a dense buffer or straight into a paged KV pool;
 *                        with a per-chunk delta it relocates already-rotated
 *                        keys and adds a (removal) patch (Sec. 5, Table evict);
 *   kamera_shift         K' = R(delta) K, in place, for keys that are already
 *                        rotated (R(delta) R(p) = R(p + delta), Sec. 1 and 3:
 *                        reorder, sliding-window survivors, Sec. 5);
 *   kamera_scatter_paged a bit copy of dense token rows into the pool slots a
 *                        page table names (the clean-view overwrite, App. E),
 *   kamera_gather_paged  and the copy back from the pool into dense rows;
 *   kamera_form_patch    the compile step's truncated SVD of given deficits
 *                        (App. A), also as one orbit patch over orderings
 *                        (Sec. 5, reorder).
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *     library never allocates, frees or synchronises; a call enqueues its
 *     kernel (kamera_form_patch: two, one after the other) on `stream` (a
 *     hipStream_t; NULL = the default stream) and returns.  Results are
 *     visible to later work on that stream.
 *   - KV rows are bf16.  Strides are in ELEMENTS (bf16) unless named _bytes;
 *     the innermost (column) stride is always 1.  Row starts must be 16-byte
 *     aligned: base pointers 16-byte aligned and every stride a multiple of 8.
 *   - Per-chunk integers (positions, deltas, row bases, token counts, page
 *     tables) are int32 arrays in device memory.
 *   - Return value: KAMERA_OK (0) or a negative kamera_status.  Argument
 *     errors are detected on the host BEFORE any HIP call, so a failed call
 *     has no side effect; kamera_last_error() then describes the problem.
 *   - Calls are thread-safe; the error text is per thread.
 *   - Contents of device arrays (page-table entries, positions) cannot be
 *     checked on the host.  Page numbers outside [0, n_pool_pages) are
 *     skipped by the kernels and flagged in the optional `status` word
 *     (bit KAMERA_STATUS_BAD_PAGE), never written out of bounds.  A page
 *     table must be injective for the result to be defined;
 *     kamera_check_page_table() verifies a host copy.
 */
#ifndef KAMERA_H
#define KAMERA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KAMERA_ABI_VERSION 4

/* Largest patch rank m accepted (>= the 128-wide head, so a full-rank patch
 * that reproduces any Delta K exactly can be applied). */
#define KAMERA_MAX_RANK 128
/* Rotated band width limit and row width limit, in elements. */
#define KAMERA_MAX_ROPE_DIM 128
#define KAMERA_MAX_HEAD_DIM 4096

typedef enum {
  KAMERA_OK = 0,
  KAMERA_ERR_NULL = -1,        /* a required pointer is NULL                    */
  KAMERA_ERR_SHAPE = -2,       /* inconsistent sizes, bands or sections         */
  KAMERA_ERR_ALIGN = -3,       /* pointer or stride breaks 16-byte row alignment */
  KAMERA_ERR_RANGE = -4,       /* a size or rank beyond the supported maximum    */
  KAMERA_ERR_ALIAS = -5,       /* an output overlaps an input it must not        */
  KAMERA_ERR_UNSUPPORTED = -6, /* a valid request this library does not implement */
  KAMERA_ERR_HIP = -7          /* the HIP runtime refused the launch             */
} kamera_status;

/* bits of the optional device status word */
#define KAMERA_STATUS_BAD_PAGE 1u

typedef enum {
  KAMERA_PAIR_NEOX = 0,        /* pair j = columns (j, j + rope_dim/2)          */
  KAMERA_PAIR_INTERLEAVED = 1  /* pair j = columns (2j, 2j + 1)                 */
} kamera_pairing;

typedef enum {
  KAMERA_SECTIONS_BLOCKED = 0,     /* pairs [0,s0) use t, [s0,s0+s1) h, rest w  */
  KAMERA_SECTIONS_INTERLEAVED = 1  /* pairs cycle t,h,w, skipping a coordinate
                                      whose section count is used up            */
} kamera_section_order;

typedef enum {
  KAMERA_POS_LINEAR = 0,   /* token i at p0 + i on every coordinate;
                              chunk_pos[c*3 + 0] = p0                         */
  KAMERA_POS_GRID3 = 1,    /* token i at (t0, h0 + i / grid_w, w0 + i % grid_w);
                              chunk_pos[c*3 + 0..2] = (t0, h0, w0)            */
  KAMERA_POS_EXPLICIT = 2  /* token i of chunk c at explicit_pos[c*explicit_
                              chunk_stride + i*3 + (0,1,2)]                   */
} kamera_pos_mode;

/* Which rehydrate kernel a call uses.  Both compute the same bits.
 * PER_HEAD: one workgroup per (plane, chunk, layer, head, token block, column
 * block); any row layout.  ROW_GROUP: one workgroup per (plane, chunk, layer,
 * token block) taking every head of a token row, so that a 16-token pool page
 * is written as one contiguous run; possible for rows of <= 8 heads of 128
 * columns (one block per head, the rope band if any being the whole head),
 * rank <= 64 in whole 16-byte U chunks, linear or grid positions (with or
 * without relocation), and byte offsets below 2^31 within one (chunk, layer)
 * slab or one layer of the pool.  A row-group workgroup takes 8 heads (one per CU),
 * or 4 (two per CU; rows of <= 4 heads, or 8 heads in two groups).  AUTO
 * takes ROW_GROUP4 where it was measured faster on MI355X: rows of 4 or 8
 * heads, chunks of >= 256 tokens and >= 2^19 rows in all (planes x chunks x
 * layers x tokens x heads), except dense outputs at rank <= 32 with 2^21 to
 * 2^23 rows.  Those, fewer rows, shorter chunks and other head counts keep
 * PER_HEAD.  A ROW_GROUP or ROW_GROUP4 request that is not possible falls
 * back to PER_HEAD. */
typedef enum {
  KAMERA_KERNEL_AUTO = 0,
  KAMERA_KERNEL_PER_HEAD = 1,
  KAMERA_KERNEL_ROW_GROUP = 2,   /* 8 heads per workgroup (4 for rows of <= 4) */
  KAMERA_KERNEL_ROW_GROUP4 = 3   /* 4 heads per workgroup, also for wider rows */
} kamera_kernel_choice;

/* How the row-group kernel spreads its work over the device (same bits
 * either way).  PERSISTENT: one resident wave of workgroups, each walking an
 * equal share (in bytes moved) of its (plane, head group)'s 16-token tiles,
 * so that a unit's set-up (W^T, page numbers) is paid once per long range
 * and every workgroup finishes together.  BLOCKS: one workgroup per token
 * block of one (plane, chunk, layer, head group), blocks of up to 1024 tokens
 * shrunk (to >= 64) until the launch has 4096 of them (2048 with 8-head
 * groups), handed out by the hardware as workgroups finish.  AUTO takes
 * BLOCKS where those blocks stay >= 512 tokens (long launches, where it
 * measured faster) and PERSISTENT otherwise, or whenever max_workgroups > 0.
 * The per-head kernel ignores the field. */
typedef enum {
  KAMERA_SCHEDULE_AUTO = 0,
  KAMERA_SCHEDULE_PERSISTENT = 1,
  KAMERA_SCHEDULE_BLOCKS = 2
} kamera_row_schedule;

typedef enum {
  KAMERA_PATCH_PRE_ROPE = 0,  /* K' = R(pos)(K + U W): the patch lives in the
                                 stored, position-free frame (Sec. 3)         */
  KAMERA_PATCH_POST_ROPE = 1  /* K' = R(pos) K + U W: the literal form of
                                 Eq. eq:operator, and the frame of a key
                                 deficit taken against R(pos) K as App. A's
                                 compile step does (see kamera_form_patch)    */
} kamera_patch_frame;

/* RoPE variant (Sec. 3 content | RoPE split; Fig. fig:unify for M-RoPE).
 * Pair j has frequency theta^(-2j/rope_dim) and rotates by angle
 * coord(j) * frequency, x' = x cos - y sin, y' = x sin + y cos. */
typedef struct {
  double theta;            /* rotary base, > 1                                */
  int32_t rope_offset;     /* first rotated column (0 for GQA/MHA, 512 MLA)  */
  int32_t rope_dim;        /* rotated width: even, <= KAMERA_MAX_ROPE_DIM    */
  int32_t pairing;         /* kamera_pairing                                 */
  int32_t n_sections;      /* 1: 1-D RoPE (coordinate t); 3: (t, h, w)       */
  int32_t sections[3];     /* pair counts of t, h, w; sum = rope_dim / 2     */
  int32_t section_order;   /* kamera_section_order                           */
} kamera_rope;

/* One stream of rows the call rebuilds: the keys (rotate = 1) or the values
 * (rotate = 0).  Element (c, l, i, h, col) of the input sits at
 *   in + c*in_stride[0] + l*in_stride[1] + i*in_stride[2] + h*in_stride[3] + col.
 * The patch factors of (c, l, h): U is n x m (token i, rank k) at
 *   U + c*u_stride[0] + l*u_stride[1] + h*u_stride[2] + i*u_stride[3] + k,
 * W is m x patch_dim at
 *   W + c*w_stride[0] + l*w_stride[1] + h*w_stride[2] + k*w_stride[3] + col',
 * col' = col - patch_offset.  A stride of 0 shares a factor (e.g. one basis
 * per layer for every chunk).  m = 0 disables the patch (U, W may be NULL).
 *
 * A plane covers the columns [col_begin, col_end) of the row (both 0: the
 * whole row; otherwise multiples of 32).  Two planes over the same rows with
 * disjoint column ranges give one row two patches of different rank, e.g. the
 * MLA latent (rank m) and the small extra patch on its rope key band that
 * Sec. 3 adds to close the latent-only residual.
 *
 * layer_rank (optional device int32 [n_layers]) lowers the rank per layer:
 * layer l uses the first min(layer_rank[l], m) ranks, 0 = no patch at that
 * layer -- the deep-half patch that stores factors for the deepest layers
 * only (Sec. 1 contributions, Table menu). */
typedef struct {
  const void* in;
  int64_t in_stride[4];
  void* out;               /* dense or pool base, see kamera_rehydrate_args  */
  int64_t out_stride[4];
  const void* U;
  int64_t u_stride[4];
  const void* W;
  int64_t w_stride[4];
  int32_t m;               /* patch rank, 0 .. KAMERA_MAX_RANK               */
  int32_t rotate;          /* 1: rotate the rope band (keys); 0: values      */
  int32_t patch_offset;    /* patched columns [patch_offset,                 */
  int32_t patch_dim;       /*                  patch_offset + patch_dim)     */
  int32_t col_begin;       /* columns this plane covers (0, 0: all)          */
  int32_t col_end;
  const int32_t* layer_rank;
} kamera_plane;

/* kamera_rehydrate -- Eq. eq:operator with the patch in the stored frame;
 * the serve step of App. A for every (chunk, layer, KV head) at once.
 *
 * Output destination of token i of chunk c, layer l, head h:
 *   dense (paged = 0): out + c*out_stride[0] + l*out_stride[1]
 *                          + (row_base[c] + i)*out_stride[2] + h*out_stride[3]
 *                      (row_base NULL = 0 for every chunk)
 *   paged (paged = 1): slot = page_table[c*pt_stride + i/page_size]*page_size
 *                             + i % page_size,
 *                      out + l*out_stride[1] + slot*out_stride[2]
 *                          + h*out_stride[3]   (out_stride[0] unused)
 * Outputs must not overlap inputs (checked on the extents the host-visible
 * sizes imply), except exactly in place: a dense output with row_base NULL,
 * the same base pointer and the same strides as the input (each element is
 * then read and written by the same workgroup; two planes in place on one
 * tensor must cover disjoint columns).  The two planes' outputs must not
 * overlap each other either, except (a) one tensor through the same mapping
 * on disjoint columns, or (b) interleaved rows: the same out_stride, all of
 * them >= 0, the layer (and for dense output the chunk) stride a multiple of
 * the row stride out_stride[2], and the bases d elements apart with
 * span <= |d| and |d| + span <= out_stride[2], span = (n_heads - 1) *
 * out_stride[3] + head_dim -- e.g. a pool [layer][slot][K|V][head][dim] in
 * which the K and V rows of a slot are adjacent, so that a page of both
 * planes is one contiguous run.  By the same rule a dense output may
 * interleave with the other plane's input (one tensor [chunk][layer][token]
 * [K|V][head][dim] rehydrated in place, each plane exactly in place).
 *
 * Relocation (delta != NULL, device int32 [n_chunks][3]): the input keys are
 * already rotated, at target - delta (survivors of a window slide, Sec. 5),
 * and the rotated planes compute
 *   K' = R(delta) K + R(target) U W      (KAMERA_PATCH_PRE_ROPE), or
 *   K' = R(delta) K + U W                (KAMERA_PATCH_POST_ROPE),
 * i.e. the move of kamera_shift fused with a (removal) patch (Sec. 5, Table
 * evict); target positions come from pos_mode as usual.  Unrotated planes
 * (values, latents) are unaffected by delta. */
typedef struct {
  int32_t n_chunks;
  int32_t n_layers;
  int32_t n_heads;             /* KV heads (1 for an MLA latent row)          */
  int32_t head_dim;            /* row width in elements, multiple of 32       */
  int32_t n_tokens;            /* tokens per chunk (the maximum if ragged)     */
  const int32_t* chunk_tokens; /* device [n_chunks] (<= n_tokens) or NULL      */
  int32_t patch_frame;         /* kamera_patch_frame                           */
  kamera_rope rope;
  int32_t pos_mode;            /* kamera_pos_mode                              */
  const int32_t* chunk_pos;    /* device [n_chunks][3] (LINEAR, GRID3)         */
  int32_t grid_w;              /* GRID3 tokens per grid row, > 0               */
  const int32_t* explicit_pos; /* device (EXPLICIT)                            */
  int64_t explicit_chunk_stride;
  int32_t n_planes;            /* 1 (keys only, e.g. MLA) or 2 (keys, values)  */
  kamera_plane plane[2];
  int32_t paged;
  const int32_t* row_base;     /* dense: device [n_chunks] or NULL             */
  const int32_t* page_table;   /* paged: device [n_chunks][pt_stride]          */
  int32_t pt_stride;
  int32_t page_size;
  int32_t n_pool_pages;
  uint32_t* status;            /* optional device word, bits OR-ed in          */
  const int32_t* delta;        /* optional: relocation of rotated keys         */
  int32_t kernel;              /* kamera_kernel_choice (0: AUTO)               */
  int32_t max_workgroups;      /* row-group kernel, persistent schedule: 0 =
                                  one resident wave of workgroups on the whole
                                  device, > 0 = at most this many (leaves CUs
                                  to concurrent work); same results.  Not
                                  allowed with KAMERA_SCHEDULE_BLOCKS
                                  (KAMERA_ERR_SHAPE).  The per-head kernel
                                  launches one workgroup per task and ignores
                                  it.                                         */
  int32_t schedule;            /* kamera_row_schedule (0: AUTO)                */
} kamera_rehydrate_args;

/* kamera_shift -- K' = R(delta_c) K in place on the rope band of every token
 * of every listed chunk (Sec. 1, Sec. 3; survivors of a window slide, Sec. 5).
 * Columns outside the band and the values are never touched.
 * delta: device [n_chunks][3] int32, the move of (t, h, w); 1-D RoPE reads
 * delta[c*3 + 0].  Token i of chunk c is row
 *   dense: k + c*k_stride[0] + l*k_stride[1] + (row_base[c] + i)*k_stride[2]
 *            + h*k_stride[3]          (row_base NULL = 0)
 *   paged: k + l*k_stride[1] + slot*k_stride[2] + h*k_stride[3],
 *          slot as in kamera_rehydrate. */
typedef struct {
  int32_t n_chunks;
  int32_t n_layers;
  int32_t n_heads;
  int32_t head_dim;
  int32_t n_tokens;
  const int32_t* chunk_tokens;
  kamera_rope rope;
  const int32_t* delta;
  void* k;
  int64_t k_stride[4];
  int32_t paged;
  const int32_t* row_base;
  const int32_t* page_table;
  int32_t pt_stride;
  int32_t page_size;
  int32_t n_pool_pages;
  uint32_t* status;
} kamera_shift_args;

/* kamera_scatter_paged / kamera_gather_paged -- bit-exact copies between
 * dense token rows and a paged pool (the copy half of the conditioning
 * switch, App. E: the clean view is restored by a plain copy; the pool is the
 * paged KV store the serve step writes into, Sec. 6).  For token i of chunk
 * c, layer l the dense row is
 *   rows + c*rows_stride_bytes[0] + l*rows_stride_bytes[1] + i*rows_stride_bytes[2]
 * and the pool row pool + l*pool_stride_bytes[0] + slot*pool_stride_bytes[1],
 * slot as in kamera_rehydrate; row_bytes bytes move, dense -> pool (scatter)
 * or pool -> dense (gather).  row_bytes and all strides: multiples of 16. */
typedef struct {
  int32_t n_chunks;
  int32_t n_layers;
  int32_t n_tokens;
  const int32_t* chunk_tokens;
  int64_t row_bytes;
  void* rows;
  int64_t rows_stride_bytes[3];
  void* pool;
  int64_t pool_stride_bytes[2];
  const int32_t* page_table;
  int32_t pt_stride;
  int32_t page_size;
  int32_t n_pool_pages;
  uint32_t* status;
} kamera_scatter_args;

/* kamera_form_patch -- the compile step of App. A on given deficits: for
 * every (chunk, layer, head) unit, the top-m singular triplets of
 * Delta (n x dim, fp32) as the stored patch
 *   U = U_svd[:, :m] * S[:m]   (n x m, bf16, singular values folded in),
 *   W = Vt[:m]                 (m x dim, bf16),
 * so U W is the best rank-m approximation of Delta.  The conditioned forward
 * pass that produces Delta needs model weights and is not part of this
 * library.
 * Frame of the factors: U W lives in the frame Delta was taken in, and the
 * kamera_rehydrate call that applies it must use the same frame.
 *   - App. A takes the key deficit against the canonical keys already turned
 *     to the target, Delta = K_cond - R(p) K: the rotated frame.  Such
 *     factors are applied with KAMERA_PATCH_POST_ROPE, K' = R(p) K + U W, at
 *     the positions p they were formed at.
 *   - For the default KAMERA_PATCH_PRE_ROPE, K' = R(p)(K + U W), turn each
 *     token's deficit back first, Delta_i <- R(-p_i) Delta_i (row i at its
 *     position p_i); the patch formed from that serves every position.
 *   Applying rotated-frame factors with KAMERA_PATCH_PRE_ROPE rotates the
 *   patch a second time and gives wrong keys.  Values and the MLA latent are
 *   never rotated, so for them the two frames coincide.
 * Layouts: element (c, l, h, i, j) of Delta at delta + c*delta_stride[0] +
 * l*delta_stride[1] + h*delta_stride[2] + i*delta_stride[3] + j (fp32,
 * 16-byte aligned rows); U and W as in kamera_plane (bf16); sigma (optional,
 * fp32) receives S[:m] at sigma + c*sigma_stride[0] + l*sigma_stride[1] +
 * h*sigma_stride[2] + k.  Method: the Gram matrix Delta^T Delta in fp32,
 * then its m largest eigenpairs, by one of two fp32 solvers:
 *   sweeps = 0 (default): Householder reduction to tridiagonal form,
 *     multisection on Sturm counts for the eigenvalues, twisted
 *     factorisation for their eigenvectors (close eigenvalues, within 1e-3 of
 *     the spectral norm, reorthogonalised), back-transformation;
 *   sweeps > 0: block cyclic Jacobi, at most `sweeps` sweeps, stopping once
 *     the off-diagonal mass is negligible (12 reach the fp32 floor here).
 * Either way singular vectors are accurate to ~1e-5 relative where the
 * spectrum has a gap at m.  W = V_m^T (bf16) is written first; U = Delta W^T
 * is then formed from that stored W in a second launch on the same stream
 * (Delta enters as a two-part bf16 split, ~2^-16 relative), so that U W is
 * the projection onto exactly the kept W.
 * Orbit patch (Sec. 5, reorder): with n_orbit = K >= 2 the deficits of K
 * orderings of the same chunk set, at delta + o*orbit_stride (o < K), are
 * averaged (fp32) and the mean is truncated as above: the one rank-m patch
 * with the least total squared error over those orderings.  A held-out
 * ordering is simply not passed.  n_orbit 0 or 1 = a single deficit.
 * U, W and sigma must not overlap the deficits, nor U overlap W
 * (KAMERA_ERR_ALIAS). */
#define KAMERA_FORM_MAX_DIM 128
typedef struct {
  int32_t n_chunks;
  int32_t n_layers;
  int32_t n_heads;
  int32_t n_tokens;            /* rows n of each Delta                          */
  int32_t dim;                 /* columns: multiple of 4, <= KAMERA_FORM_MAX_DIM */
  int32_t m;                   /* rank kept: 1 .. dim                           */
  int32_t sweeps;              /* 0 = tridiagonal solver, > 0 = Jacobi limit   */
  int32_t n_orbit;             /* deficits averaged per unit (0 or 1 = one)     */
  const float* delta;
  int64_t delta_stride[4];
  void* U;
  int64_t u_stride[4];
  void* W;
  int64_t w_stride[4];
  float* sigma;
  int64_t sigma_stride[3];
  int64_t orbit_stride;        /* elements between orbit members of delta       */
  int32_t* sweeps_done;        /* optional: Jacobi sweeps each unit ran (0 with
                                  the tridiagonal solver), dense
                                  [n_chunks][n_layers][n_heads] int32          */
} kamera_form_args;

int kamera_rehydrate(const kamera_rehydrate_args* args, void* stream);
int kamera_form_patch(const kamera_form_args* args, void* stream);
int kamera_shift(const kamera_shift_args* args, void* stream);
int kamera_scatter_paged(const kamera_scatter_args* args, void* stream);
int kamera_gather_paged(const kamera_scatter_args* args, void* stream);

/* Host-side check of a page table copy (host memory, n_chunks x pt_stride,
 * the first ceil(tokens/page_size) entries of each row are used): every used
 * entry in [0, n_pool_pages) and no page used twice.  Returns KAMERA_OK or
 * KAMERA_ERR_RANGE (out of range) / KAMERA_ERR_ALIAS (duplicate). */
int kamera_check_page_table(const int32_t* host_page_table, int32_t n_chunks,
                            int32_t pt_stride, int32_t n_tokens,
                            int32_t page_size, int32_t n_pool_pages);

/* Run exactly the host-side checks of an entry point (0 kamera_rehydrate,
 * 1 kamera_shift, 2 kamera_scatter_paged, 3 kamera_gather_paged,
 * 4 kamera_form_patch) on `args` without launching anything: KAMERA_OK when
 * the call would be enqueued, else the error code the call would return.
 * Touches no device memory. */
int kamera_validate(int32_t which, const void* args);

/* Which kernel kamera_rehydrate would launch for `args` (see
 * kamera_kernel_choice), after exactly its host-side checks:
 * KAMERA_PLAN_PER_HEAD, KAMERA_PLAN_ROW_GROUP (8 heads per workgroup),
 * KAMERA_PLAN_ROW_GROUP4 (4 heads per workgroup), KAMERA_PLAN_NONE for a call
 * with nothing to do, or the negative error code the call would return.  A
 * positive plan equals the kamera_kernel_choice that requests that kernel.
 * Touches no device memory. */
#define KAMERA_PLAN_NONE 0
#define KAMERA_PLAN_PER_HEAD 1
#define KAMERA_PLAN_ROW_GROUP 2
#define KAMERA_PLAN_ROW_GROUP4 3
int kamera_rehydrate_plan(const kamera_rehydrate_args* args);

/* How the row-group kernel would spread a kamera_rehydrate call for `args`
 * (see kamera_row_schedule), after exactly its host-side checks:
 * KAMERA_SCHEDULE_PERSISTENT or KAMERA_SCHEDULE_BLOCKS; 0 when the call runs
 * the per-head kernel or has nothing to do; else the negative error code the
 * call would return.  Touches no device memory. */
int kamera_rehydrate_schedule(const kamera_rehydrate_args* args);

/* Text of the last error on the calling thread ("" after a successful call);
 * valid until the next call on that thread. */
const char* kamera_last_error(void);
int kamera_abi_version(void);
/* sizeof of the argument structs: 0 rehydrate, 1 shift, 2 scatter, 3 plane,
 * 4 rope, 5 form; -1 otherwise.  Lets a foreign-function binding check its
 * layout. */
int64_t kamera_struct_size(int32_t which);

#ifdef __cplusplus
}
#endif

#endif /* KAMERA_H */
