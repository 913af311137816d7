/*
 * memfine.h - C ABI of the MI355X (gfx950) chunked MoE expert layer.
 *
 * The layer is the per-GPU hot path of MemFine (memory-aware fine-grained
 * scheduling for MoE training): on one GPU's share of expert-parallel work it
 * runs dispatch (group the received token-slots by local expert), the expert
 * SwiGLU FFN on every expert's rows, and the gate-weighted combine, over C
 * contiguous token chunks (paper Section 4.1, Eq. (6)); the backward
 * recomputes each chunk before back-propagating it (Eq. (7)).  C comes from
 * the paper's activation-memory model (Section 4.2, Eq. (8), Eq. (9), bins).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers named d_* are device pointers, h_* host pointers.  Every buffer
 *   is owned by the caller; the library keeps no state between calls except a
 *   lazily created per-process profiling table; the launch options of
 *   memfine_set_launch_options (one process-wide setting); for calls made
 *   with a NULL allocator, one workspace block per (device, stream), carved
 *   into each chunk's buffers and reused by the next chunk in stream order
 *   (grown from a per-device stream-ordered pool when a call needs more,
 *   kept until memfine_workspace_trim or the end of the process: see
 *   memfine_workspace_held); one pinned host buffer of 1025 ints per device
 *   for memfine_count; and, only when the side-stream launch option is on,
 *   two side streams and three events per device (kept until the process
 *   ends).
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Device work is enqueued asynchronously on it; only memfine_count and
 *   memfine_profile_end synchronise (with the stream / the recorded events).
 * - Return value: MEMFINE_OK (0) or a negative status.  Argument errors are
 *   detected on the host and returned before anything is enqueued.  A HIP
 *   failure returns MEMFINE_ERR_HIP; an allocator that returns NULL gives
 *   MEMFINE_ERR_OOM.  After a failed call the outputs are unspecified, and
 *   every internal allocation has been handed back.
 * - Shapes (memfine_shape): T received tokens, h hidden size, F expert FFN
 *   size (g_e in the paper), E local experts, k slots per token (top-k).
 *   Requirements: T >= 0, T*k < 2^31, h % 64 == 0, F % 64 == 0, h, F >= 64,
 *   1 <= k, 1 <= E <= 1024.
 * - Layouts, all row-major and contiguous:
 *     idx    int32 [T, k]       expert of each slot, 0 <= idx < E
 *     gates  float [T, k]       score of each slot (need not sum to 1)
 *     X, Y, dY, dX   dtype [T, h]
 *     W1     dtype [E, 2F, h]   rows 0..F-1: SiLU gate, rows F..2F-1: up
 *     W2     dtype [E, h, F]
 *     dW1, dW2  float, shaped like W1, W2;   dgates float [T, k]
 *   dtype is bf16 (MEMFINE_BF16, raw 16-bit storage) or float (MEMFINE_F32).
 *   Per slot (token t, slot j, expert e = idx[t,j], g = gates[t,j]):
 *     u = W1[e] X[t];  a = silu(u[0:F]) * u[F:2F];  Y[t] += g * (W2[e] a).
 *   Arithmetic: fp32 accumulation everywhere; on the bf16 path the per-chunk
 *   intermediates are stored as bf16.
 */
#ifndef MEMFINE_H
#define MEMFINE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define MEMFINE_OK                0
#define MEMFINE_ERR_INVALID_ARG  (-1)
#define MEMFINE_ERR_UNSUPPORTED  (-2)
#define MEMFINE_ERR_BUDGET       (-3)
#define MEMFINE_ERR_OOM          (-4)
#define MEMFINE_ERR_HIP          (-5)
#define MEMFINE_ERR_SCRATCH      (-6)

/* element types */
#define MEMFINE_BF16  0
#define MEMFINE_F32   1

/* passes for memfine_workspace_bytes */
#define MEMFINE_PASS_FWD  0
#define MEMFINE_PASS_BWD  1

typedef struct memfine_shape {
  int64_t T;      /* received tokens (rows of X)                       */
  int32_t h;      /* hidden size                                        */
  int32_t F;      /* expert FFN size (SwiGLU width; FC1 has 2F rows)    */
  int32_t E;      /* local experts                                      */
  int32_t k;      /* slots per token (top-k)                            */
  int32_t dtype;  /* MEMFINE_BF16 or MEMFINE_F32                        */
} memfine_shape;

/*
 * Optional device-memory provider for the per-chunk working buffers.
 * alloc(bytes, stream, ctx) returns a device pointer (256-byte aligned) that
 * is usable in stream order on `stream`, or NULL on failure; release(ptr,
 * bytes, stream, ctx) gives it back in stream order.  When the allocator
 * argument of a call is NULL the library takes the chunk's buffers from its
 * cached workspace block for the call's stream (see the conventions above):
 * the block's size is the largest per-chunk workspace asked for on that
 * stream since it was last trimmed, and it stays allocated after the call
 * returns (memfine_workspace_held / memfine_workspace_trim).
 */
typedef struct memfine_allocator {
  void* (*alloc)(size_t bytes, void* stream, void* ctx);
  void (*release)(void* ptr, size_t bytes, void* stream, void* ctx);
  void* ctx;
} memfine_allocator;

/* Output of the planner (all fields filled on MEMFINE_OK and on
 * MEMFINE_ERR_BUDGET). */
typedef struct memfine_plan_info {
  int64_t s_recv;        /* s'': received slots, the sum of the counts      */
  int64_t beta;          /* bytes per received slot used by Eq. (8)         */
  int64_t avail;         /* budget - fixed, the numerator of Eq. (8)        */
  double s_max;          /* Eq. (8): avail / beta (for reporting only)      */
  int64_t c_theory;      /* Eq. (9): ceil(s'' / s'_max); -1 if avail <= 0   */
  int32_t chunks;        /* chosen chunk count (a bin)                      */
  int32_t fits;          /* 1 if the call returned MEMFINE_OK               */
  int64_t paper_peak_bytes; /* beta_paper * slots of the largest chunk      */
  int64_t beta_paper;    /* Table 2 rows 11-13: D_t (2h + 2F)               */
  int64_t beta_impl;     /* this library's backward bytes per slot          */
  int64_t workspace_bytes; /* memfine_workspace_bytes(chunks, backward)     */
  int32_t paper_chunks;  /* the bin Eq. (8)/(9) give with beta_paper alone  */
  int32_t reserved;
} memfine_plan_info;

/*
 * Launch options, for measurements and tests.  Every GEMM setting (tile,
 * raster, split_tail, pair, streams) gives bit-identical results (each
 * output element is one lane's fp32 sum in increasing K order whatever the
 * tiling); chunk_order changes the order of the sums that form Y and dX.
 * Process-wide; a layer call reads them once when it starts, and
 * memfine_workspace_bytes (hence memfine_plan) follows chunk_order.
 */
#define MEMFINE_TILE_AUTO    0   /* per problem (the default)                  */
#define MEMFINE_TILE_128     1   /* 128 x 128 tiles, 4 waves                   */
#define MEMFINE_TILE_256     2   /* 256 x 256 tiles, 8 waves, direct copies    */
#define MEMFINE_TILE_256_REG 3   /* 256 x 256 tiles, 8 waves, register-staged  */
/*
 * Chunk order.  MEMFINE_CHUNK_TOKENS (the default) is the paper's split,
 * Eq. (6): chunk i holds the slots of tokens [i T / C, (i + 1) T / C).
 * MEMFINE_CHUNK_EXPERTS, a variant that is not in the paper: one dispatch
 * groups all T k slots by expert, and chunk c holds rows [c N / C,
 * (c + 1) N / C) of that grouping (N = T k), i.e. a run of whole experts
 * with at most the first and last split.  An expert's weights are then read,
 * and its fp32 dW written, in one chunk (two for a split expert) instead of
 * in every chunk; in exchange Y and dX are sums over chunks: the chunk that
 * holds a token's first row writes its partial sum, later chunks add theirs
 * to the stored value (one rounding to the storage type per chunk), so
 * these two outputs are not bit-identical across C or to the token order,
 * while dW, dgates and the per-chunk peak (at most ceil(N / C) rows plus
 * the layer's routing tables) follow the same definitions.
 */
#define MEMFINE_CHUNK_TOKENS  0
#define MEMFINE_CHUNK_EXPERTS 1
typedef struct memfine_launch_options {
  int32_t tile;        /* MEMFINE_TILE_*                                       */
  int32_t raster;      /* -1 per problem; 0 row-major by workgroup id; 1..3
                          XCD blocks with groups of 4, 8, 16 m-tiles; 4 XCD
                          blocks row-major                                     */
  int32_t split_tail;  /* 1: a short last round of a GEMM runs as quarter tiles */
  int32_t pair;        /* 1: FC1 dgrad and FC1 wgrad in one launch             */
  int32_t streams;     /* 1: the weight gradients on two side streams          */
  int32_t chunk_order; /* MEMFINE_CHUNK_* (changes results: see above)         */
} memfine_launch_options;

/* NULL restores the defaults {AUTO, -1, 1, 0, 0, TOKENS}.
 * MEMFINE_ERR_INVALID_ARG on a value out of range (the setting is then
 * unchanged). */
int memfine_set_launch_options(const memfine_launch_options* opts);
int memfine_get_launch_options(memfine_launch_options* opts_out);

/*
 * Expert counts over all T tokens: the "first notification" of the paper's
 * Section 4.2 that delivers the number of received slots s''.
 *   d_idx     int32 [T, k] device
 *   d_work    int32 [E + 1] device scratch owned by the caller; on return
 *             d_work[e] = slots routed to expert e and d_work[E] = number of
 *             ids outside [0, E)
 *   h_counts  int64 [E] host output
 * Synchronises `stream`.  Returns MEMFINE_ERR_INVALID_ARG when any id is out
 * of range (h_counts then counts only the valid ids).
 */
int memfine_count(const memfine_shape* shape, const int32_t* d_idx, int32_t* d_work,
                  int64_t* h_counts, void* stream);

/*
 * Dispatch of one chunk, tokens [t0, t1) (the "dispatch" of Eq. (4)), exposed
 * so that tests can check the exact permutation the layer uses.  With
 * n = (t1 - t0) * k and global slot id s = t * k + j:
 *   d_counts       int32 [E]       slots of expert e in the chunk
 *   d_offsets      int32 [E + 1]   exclusive prefix sum, d_offsets[E] = n
 *   d_sorted_slot  int32 [n]       slot ids grouped by expert; ascending
 *                                  slot id inside an expert (stable)
 *   d_row_of_slot  int32 [n]       row of slot t0*k + i in that order
 * Precondition: ids already validated (memfine_count).  Scratch comes from
 * `alloc` (NULL = the library's workspace block for the stream).  Asynchronous.
 */
int memfine_dispatch(const memfine_shape* shape, const int32_t* d_idx, int64_t t0, int64_t t1,
                     int32_t* d_counts, int32_t* d_offsets, int32_t* d_sorted_slot,
                     int32_t* d_row_of_slot, const memfine_allocator* alloc, void* stream);

/*
 * Memory-aware chunk tuning (paper Section 4.2).  Pure host arithmetic, exact
 * in integers.
 *   h_counts      int64 [E]   slots per local expert (memfine_count)
 *   budget_bytes  the numerator of Eq. (8): memory left for this layer's
 *                 chunked MoE activations (alpha*M_GPU - M_sta - non-MoE)
 *   fixed_bytes   subtracted from the budget first (>= 0)
 *   beta_bytes    bytes per received slot, see below
 *   bins, nbins   allowed chunk counts (each >= 1), e.g. {1, 2, 4, 8}
 * Chooses s'' = sum(counts), s'_max = (budget - fixed) / beta (Eq. (8)),
 * c = ceil(s'' / s'_max) (Eq. (9)), then the smallest bin >= c (decided
 * exactly as bin * (budget - fixed) >= s'' * beta).
 *   beta_bytes > 0: that beta; the paper's model alone decides.
 *   beta_bytes = 0 (default): beta = max(beta_paper, beta_impl), the larger
 *     of Table 2 rows 11-13, D_t (2h + 2F), and this library's own backward
 *     bytes per slot; then, so that Eq. (3) holds for the memory the layer
 *     really takes, the chosen bin moves up to the next bin while
 *     memfine_workspace_bytes(bin, backward) > budget - fixed (the rounding
 *     of the chunk split and the per-chunk metadata are not in Eq. (9)).
 *     On MEMFINE_OK the chunk's workspace therefore fits the budget.
 * If no bin is large enough, or budget - fixed <= 0, *chunks_out = the
 * largest bin and the call returns MEMFINE_ERR_BUDGET.  s'' = 0 gives the
 * smallest bin.  `info` may be NULL; info->paper_chunks reports the bin that
 * the paper's beta alone would give.
 */
int memfine_plan(const memfine_shape* shape, const int64_t* h_counts, int64_t budget_bytes,
                 int64_t fixed_bytes, int64_t beta_bytes, const int32_t* bins, int32_t nbins,
                 int32_t* chunks_out, memfine_plan_info* info);

/*
 * Bytes of working memory the layer allocates for its largest chunk (the
 * per-chunk buffers of memfine_moe_fwd or memfine_moe_bwd, pass =
 * MEMFINE_PASS_FWD / MEMFINE_PASS_BWD) - the activation peak of the chunked
 * layer that Section 4.1 says replaces the unchunked one.  Under
 * MEMFINE_CHUNK_EXPERTS it adds the layer's routing tables, held for the
 * whole call.  Returns < 0 on invalid arguments.
 */
int64_t memfine_workspace_bytes(const memfine_shape* shape, int32_t chunks, int32_t pass);

/*
 * The library's cached workspace block for calls with a NULL allocator
 * (paper Section 4.1: the layer's activation peak is the largest chunk's).
 * memfine_workspace_held: bytes of the block kept for (the current device,
 * `stream`); 0 if none.  memfine_workspace_trim: if that block is larger than
 * keep_bytes, it is released in stream order (after the work enqueued on
 * `stream` so far) and, when keep_bytes > 0, replaced by a block of
 * keep_bytes; afterwards the held bytes are at most keep_bytes.  A caller
 * that raises the chunk count to free memory trims to
 * memfine_workspace_bytes(new chunks, MEMFINE_PASS_BWD).  Not to be called
 * while a layer call runs on the same stream from another thread.
 */
int memfine_workspace_held(void* stream, int64_t* bytes_out);
int memfine_workspace_trim(void* stream, int64_t keep_bytes);

/*
 * High-water mark of the library's per-device stream-ordered pool (the
 * bytes its blocks held at most at once, on the current device) since the
 * pool was created or last reset (reset = 1 resets it after reading).  0
 * before the first call that needed a block.
 */
int memfine_pool_high_water(int64_t* bytes_out, int32_t reset);

/* ------------------------------------------------------------------------
 * MACT from the model configuration (paper Section 3 and Section 4.2).
 * Pure host arithmetic, exact (128-bit integers); no device state.
 *
 * The memory model uses the symbols of the paper's notation table; every
 * size is an element count and D_t the bytes per activation element.
 */
typedef struct memfine_model {
  int64_t b, s;            /* micro-batch size, sequence length                */
  int64_t h, a, h_d, k_a;  /* hidden size, heads, head dim, kv heads           */
  int64_t e_n, g_e;        /* router output width, expert FFN size (F)         */
  int32_t t, c;            /* tensor- and context-parallel sizes (>= 1)        */
  int32_t v, p;            /* pipeline stages per GPU, pipeline size (>= 1)    */
  int32_t D_t;             /* activation bytes per element (>= 1)              */
  int32_t full_recompute;  /* 1: m_g = 1; 0: m_g = v p + p - 2 r_pp - 1        */
} memfine_model;

/*
 * Eq. (1): static memory = (D_para + D_grad + 4 D_opt) * v * l * sum(S_para),
 * parameters, gradients and four optimizer-state copies of the m_n weighted
 * modules of a layer (S_para[i] elements each), v stages of l layers.
 * *bytes_out receives the total.  MEMFINE_ERR_INVALID_ARG on a negative or
 * zero size factor, a negative S_para, or a result beyond int64.
 */
int memfine_static_memory(const int64_t* S_para, int32_t m_n, int32_t v, int32_t l,
                          int32_t D_para, int32_t D_grad, int32_t D_opt, int64_t* bytes_out);

/*
 * Eq. (2): peak activation bytes at pipeline rank r_pp (0 <= r_pp < p) with
 * s_recv received slots, m_g/(t c) D_t b (s (5h + a h_d + 2 k_a h_d + e_n)
 * + s_recv (2h + 2 g_e)), rounded up to whole bytes.  With chunking, s_recv
 * is the largest chunk's slots.  MEMFINE_ERR_INVALID_ARG on invalid fields,
 * m_g < 1, or a result beyond int64.
 */
int memfine_activation_memory(const memfine_model* m, int32_t r_pp, int64_t s_recv,
                              int64_t* bytes_out);

/*
 * MACT set-up, once per pipeline rank before training: the threshold table
 * of the bins.  s'_max is Eq. (8) with alpha = alpha_num / alpha_den, GPU
 * memory M_gpu and static memory M_sta (bytes); thresholds_out[i] is the
 * largest s'' for which bins[i] chunks keep Eq. (3), floor(bins[i] * s'_max),
 * or -1 when the part of Eq. (2) that does not depend on s'' alone exceeds
 * alpha M_gpu - M_sta.  Values beyond int64 are clamped to INT64_MAX.
 */
int memfine_mact_thresholds(const memfine_model* m, int32_t r_pp, int64_t M_gpu, int64_t alpha_num,
                            int64_t alpha_den, int64_t M_sta, const int32_t* bins, int32_t nbins,
                            int64_t* thresholds_out);

/*
 * MACT at run time, per iteration and layer: the smallest bin whose
 * threshold admits the received slots s_recv (the threshold form of Eq. (9)
 * followed by the bin choice).  When no bin admits them, *chunks_out is the
 * largest bin and the call returns MEMFINE_ERR_BUDGET.
 */
int memfine_mact_select(const int32_t* bins, const int64_t* thresholds, int32_t nbins,
                        int64_t s_recv, int32_t* chunks_out);

/*
 * Chunked forward, Eq. (6): Y = concat(F_w(X_1), ..., F_w(X_C)), with
 * F_w = combine(expert(dispatch(.))) of Eq. (4) on tokens
 * [floor(i*T/C), floor((i+1)*T/C)).  Every chunk's buffers are allocated
 * before and released after its kernels.  Nothing is kept for the backward.
 * Y is overwritten.  `chunks` >= 1 (chunks > T behaves like T).  A slot whose
 * id lies outside [0, E) is dropped: it contributes nothing to Y (and, in the
 * backward, nothing to dX or dW; its dgates entry is 0).
 */
int memfine_moe_fwd(const memfine_shape* shape, int32_t chunks, const void* d_X,
                    const int32_t* d_idx, const float* d_gates, const void* d_W1,
                    const void* d_W2, void* d_Y, const memfine_allocator* alloc, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * chunked forward of memfine_moe_fwd, same arguments (no allocator) and
 * bit-identical results, with every chunk's working buffers in one static
 * device array of MEMFINE_NOALLOC_SCRATCH_BYTES (64 MiB) that the library's
 * code object carries; each GPU the library runs on holds its own copy until
 * the process ends.  The call allocates and frees nothing (no hipMalloc,
 * pool or allocator call; the array's address is looked up once per device
 * with hipGetSymbolAddress).  A call whose largest chunk needs more than the
 * array, memfine_workspace_bytes(shape, chunks, MEMFINE_PASS_FWD) >
 * MEMFINE_NOALLOC_SCRATCH_BYTES, returns MEMFINE_ERR_SCRATCH before anything
 * is enqueued: raise `chunks`.  Nothing in the array needs to start at zero
 * (every buffer is written before it is read).  All calls on one GPU share
 * its array: calls that overlap on one GPU (other streams, other threads)
 * race, and the caller must order them (e.g. one stream).
 */
#define MEMFINE_NOALLOC_SCRATCH_BYTES (64ll << 20)
int memfine_moe_fwd_noalloc(const memfine_shape* shape, int32_t chunks, const void* d_X,
                            const int32_t* d_idx, const float* d_gates, const void* d_W1,
                            const void* d_W2, void* d_Y, void* stream);

/*
 * Chunked-recompute backward, Eq. (7): for each chunk in ascending order,
 * recompute its forward, then back-propagate dY's rows of that chunk.
 * Overwrites dX and dgates.  dW1/dW2 are overwritten when accumulate_dW == 0
 * and added to when accumulate_dW == 1.
 */
int memfine_moe_bwd(const memfine_shape* shape, int32_t chunks, const void* d_X,
                    const int32_t* d_idx, const float* d_gates, const void* d_W1,
                    const void* d_W2, const void* d_dY, void* d_dX, float* d_dW1, float* d_dW2,
                    float* d_dgates, int32_t accumulate_dW, const memfine_allocator* alloc,
                    void* stream);

/* ------------------------------------------------------------------------
 * Router in front of the expert layer (Table 2 rows 9-10 store its input and
 * its logits; the gates it produces are the scores that multiply the expert
 * outputs, Table 2 "score mul").  `shape` is the layer's shape; the router
 * needs k <= 16 and k <= E <= 256 (MEMFINE_ERR_UNSUPPORTED otherwise): up to
 * the 256 routed experts of the paper's Table 3 models.
 *
 * Forward: logits = X Wr^T (fp32 accumulation), softmax over the E experts,
 * the k largest logits (equal logits: the lower expert id first), and the
 * gates renormalised over the selected k (the full softmax denominator
 * cancels, so gates_j = exp(z_j - z_max) / sum over the selected).
 *   d_X       dtype [T, h];   d_Wr  dtype [E, h]
 *   d_idx     int32 [T, k] out, largest logit first
 *   d_gates   float [T, k] out
 *   d_logits  float [T, E] out, may be NULL
 * Asynchronous.  Up to 64 logits (or E not a multiple of 32) one fused
 * kernel, no working memory; wider routers compute the logits as a grouped
 * GEMM and select from them, taking 256 bytes and, when d_logits is NULL,
 * the [T, E] fp32 logits from the library's per-stream workspace (as a
 * layer call with a NULL allocator does); MEMFINE_ERR_OOM if that fails.
 */
int memfine_router_fwd(const memfine_shape* shape, const void* d_X, const void* d_Wr,
                       int32_t* d_idx, float* d_gates, float* d_logits, void* stream);

/*
 * Backward from the expert layer's dgates (memfine_moe_bwd's output), with
 * the selection held fixed: per token, with c = sum_j g_j dg_j,
 *   dlogits[t, idx_j] = g_j (dg_j - c), 0 for the unselected experts;
 *   dX  = dlogits Wr   (accumulate_dX = 1 adds it into d_dX, e.g. the
 *                       layer's dX; 0 overwrites)
 *   dWr = dlogits^T X  (float [E, h]; accumulate_dWr as above)
 * Slots whose id lies outside [0, E) pass no gradient.  Working memory
 * (dense dlogits rows and split-K partials of dWr) comes from `alloc`.
 */
int memfine_router_bwd(const memfine_shape* shape, const void* d_X, const void* d_Wr,
                       const int32_t* d_idx, const float* d_gates, const float* d_dgates,
                       void* d_dX, float* d_dWr, int32_t accumulate_dX, int32_t accumulate_dWr,
                       const memfine_allocator* alloc, void* stream);

/* Static, human-readable text for a status code. */
const char* memfine_status_str(int status);

/*
 * Kernel timing for performance reports.  memfine_profile_begin(mask) makes
 * later calls record a pair of HIP events around every launch of the kernels
 * whose id bit is set in `mask` (ids: MEMFINE_K_*).  memfine_profile_end waits
 * for those events and returns, per kernel id, the number of launches, the
 * summed launch durations in milliseconds, and the algorithmic flops and HBM
 * bytes of those launches; then it stops recording.
 */
#define MEMFINE_K_COUNT       0
#define MEMFINE_K_DISPATCH    1
#define MEMFINE_K_FC1         2   /* forward FC1 + SwiGLU                    */
#define MEMFINE_K_FC2         3   /* forward FC2                             */
#define MEMFINE_K_COMBINE     4
#define MEMFINE_K_FC1_RECOMP  5   /* backward: FC1 recompute + SwiGLU bwd    */
#define MEMFINE_K_FC2_DGRAD   6   /* backward: dA = dY W2                    */
#define MEMFINE_K_FC2_WGRAD   7
#define MEMFINE_K_FC1_WGRAD   8
#define MEMFINE_K_FC1_DGRAD   9
#define MEMFINE_K_UNPERMUTE  10   /* dX sum over slots and gate gradient     */
#define MEMFINE_K_FC1_BWD    11   /* FC1 dgrad and FC1 wgrad in one launch   */
#define MEMFINE_K_ROUTER_FWD 12   /* router logits, softmax, top-k, gates    */
#define MEMFINE_K_ROUTER_BWD_DX 13 /* router: dz per token, dX contribution */
#define MEMFINE_K_ROUTER_WGRAD 14 /* router: split-K partials of dz^T X     */
#define MEMFINE_K_ROUTER_REDUCE 15 /* router: sum of the partials into dWr  */
#define MEMFINE_K_NUM        16

typedef struct memfine_kernel_stat {
  int64_t launches;
  double total_ms;
  double flops;   /* algorithmic floating-point operations, all launches */
  double bytes;   /* algorithmic HBM bytes, all launches                  */
} memfine_kernel_stat;

int memfine_profile_begin(uint32_t mask);
int memfine_profile_end(memfine_kernel_stat* out /* [MEMFINE_K_NUM] */);

#ifdef __cplusplus
}
#endif

#endif /* MEMFINE_H */
