/*
 * moe.h -- C ABI of the MI355X (gfx950) MoE-layer library.
 *
 * One GPU's share of an expert-parallel MoE layer (paper section 2.1, Fig 3):
 * top-k routing, dispatch of token rows into expert-contiguous buffers, a
 * per-expert SwiGLU grouped GEMM (GEMM0 = gate and up projection, SiLU times
 * up, GEMM1 = down projection) and the weighted combine.  The forward pass is
 * one persistent megakernel whose workers are split at run time into
 * data-movement workers (dispatch and combine) and MFMA compute workers
 * (section 3, section 4); an in-kernel cost model (Eq 1-16) picks the split c,
 * the chunk count K and the steal count from the routing histogram.
 *
 * On one GPU the cross-GPU dispatch and combine become HBM-to-HBM copies:
 * rows of source rank r live in the staging region x[r*Tr .. (r+1)*Tr) and
 * their outputs go to y[r*Tr .. (r+1)*Tr).  This GPU is EP rank 0 and holds
 * the local experts [first_local_expert, first_local_expert + n_local_experts).
 *
 * Conventions for every entry point
 *  - bf16 tensors are passed as uint16_t bit patterns, row-major, densely
 *    packed (no strides), in device memory.
 *  - Every pointer argument is a device pointer unless marked "host".
 *  - The caller owns all memory: inputs, outputs, packed weights and the
 *    workspace.  The library never allocates or frees device memory; the
 *    handle holds host state only.
 *  - Streams are hipStream_t passed as void* (NULL = the null stream).  Calls
 *    are asynchronous on that stream unless documented to synchronise.
 *  - A handle is used from one host thread and one stream at a time.
 *  - Argument errors are detected on the host before anything is launched
 *    and return MOE_ERR_INVALID_ARG (nothing is enqueued).  Errors detected on
 *    the device (out-of-range routing ids, a wait that timed out) are latched
 *    in a device error word and returned by moe_sync_status and by the next
 *    synchronising call.
 *  - moe_last_error() returns a thread-local message for the last failure.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct moe_handle moe_handle;

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1, /* bad argument, detected on the host */
  MOE_ERR_UNSUPPORTED = -2, /* valid but outside what the kernels support */
  MOE_ERR_HIP = -3,         /* a HIP runtime call failed */
  MOE_ERR_TIMEOUT = -4,     /* a device-side wait exceeded its time limit */
  MOE_ERR_ROUTING = -5,     /* routing ids out of range or repeated in a row */
  MOE_ERR_STATE = -6        /* call order violated (e.g. forward before tables) */
} moe_status;

typedef enum {
  MOE_MODE_DYNAMIC = 0, /* megakernel, plan from the in-kernel cost model */
  MOE_MODE_STATIC = 1,  /* megakernel, fixed split c = static_c, K = 1, no steal,
                           combine by movement workers only */
  MOE_MODE_SERIAL = 2   /* four kernels in sequence, each on every CU:
                           dispatch, GEMM0 + SiLU*up, GEMM1, combine */
} moe_mode;

/* Problem shape (section 3.1 notation: H hidden, I = ffn, E experts, top-k). */
typedef struct {
  int32_t n_src_ranks;        /* R >= 1 source ranks (staging regions) */
  int32_t tokens_per_rank;    /* Tr >= 1; T = R*Tr tokens in total */
  int32_t hidden;             /* H, multiple of 64, <= 16384 */
  int32_t ffn;                /* I (F), multiple of 64, <= 32768 */
  int32_t n_experts;          /* E, 1..512 */
  int32_t top_k;              /* k, 1..min(E, 8) */
  int32_t n_local_experts;    /* E_l, 1..64 */
  int32_t first_local_expert; /* e0, 0 <= e0 <= E - E_l */
  int32_t n_shared_experts;   /* S, 0..8, always-on experts applied to rank-0 tokens */
  int32_t n_workers;          /* persistent workgroups N; 0 = one per CU */
  int32_t gemm1_split;        /* split-K factor of GEMM1 (K = F): 1, 2, 4 or 8; 0 = chosen from F/H */
} moe_config;

#define MOE_CALIB_MAX_C 32
#define MOE_CALIB_MAX_K 4

/* Which movement work the bubble-steal window of Eq 11 holds (section
 * 3.2.2 leaves its W_comm undefined). */
typedef enum {
  MOE_WINDOW_PLAIN = 0,        /* W_dispatch + W_combine, the volume of Eq 5 */
  MOE_WINDOW_MOVE_STEAL = 1,   /* (W_dispatch + W_combine)(K-1)/K: compute workers
                                  whose GEMM0 rows are not dispatched yet copy rows
                                  themselves, so the first chunk's dispatch runs on
                                  all N workers before any GEMM tile starts, and the
                                  last chunk's combine runs on all N workers after
                                  the GEMMs (section 4); the default */
  MOE_WINDOW_LAST_COMBINE = 2  /* W_dispatch + W_combine (K-1)/K: only the last
                                  chunk's combine is outside the window */
} moe_steal_window;

/* Hardware input of the cost model (section 3, Fig 4a/b, Fig 7a).
 * For grid point i: c[i] movement workers move bw_bytes_per_s[i] payload
 * bytes/s (BW(c)) while N - c[i] compute workers reach comp_flop_per_s[i]
 * (TFLOPS(N - c)).  eff_chunk[j] is the chunked/unchunked GEMM throughput
 * ratio at k_chunks[j] chunks; alpha is the tile-level overlap ratio (Eq 6).
 * literal_volumes = 1 uses the printed remote-only volumes of Eq 2-3;
 * 0 (default) counts every moved row, since on one GPU rank 0's rows also go
 * through the movement workers.  bw_all_bytes_per_s is the rate of all N
 * workers moving together: the last chunk's combine runs on every worker
 * (section 4), so the exposed tail of Eq 6/10 moves at that rate; 0 takes the
 * printed BW(c) instead.  steal_window selects the window of Eq 11 (a
 * moe_steal_window); steal_ceil = 1 (the default) rounds Eq 14's share
 * W_steal / (N W_tile) up to whole tiles, 0 takes its whole part.  With
 * literal_volumes = 1, bw_all = 0, MOE_WINDOW_PLAIN and steal_ceil = 0 the
 * model is the printed equations as they stand. */
typedef struct {
  int32_t n_c;
  int32_t c[MOE_CALIB_MAX_C];            /* ascending, 1 <= c < N */
  double bw_bytes_per_s[MOE_CALIB_MAX_C];
  double comp_flop_per_s[MOE_CALIB_MAX_C];
  int32_t n_k;
  int32_t k_chunks[MOE_CALIB_MAX_K];     /* ascending, each in {1,2,4,8} */
  double eff_chunk[MOE_CALIB_MAX_K];     /* in (0, 1] */
  double alpha;                          /* in [0, 1] */
  int32_t literal_volumes;
  int32_t static_c;                      /* split used by MOE_MODE_STATIC */
  double bw_all_bytes_per_s;             /* >= 0; 0: tail at BW(c) */
  int32_t steal_window;                  /* a moe_steal_window */
  int32_t steal_ceil;                    /* 0 or 1 */
} moe_calib;

/* Execution plan (section 3.3): the split, the chunk count and the steal count. */
typedef struct {
  int32_t c;          /* movement workers (section 3.1) */
  int32_t K;          /* chunk count of the chunk pipeline (section 3.2.1) */
  int32_t n_steal;    /* GEMM tiles each movement worker steals (Eq 14) */
  int32_t final_all;  /* 1: every worker joins the combine once the compute
                         queue is empty (section 4); 0: movement workers only */
  double t_pred_s;    /* T_total(c, K) predicted by Eq 15; 0 for forced plans */
} moe_plan;

/* Byte offsets of the workspace regions (for inspection by tests). */
typedef struct {
  size_t total;
  size_t slot;        /* int32 [T*k]: slot of pair (g,j) or -1 */
  size_t inv;         /* int32 [T*min(k,E_l)]: g*k+j of each slot */
  size_t first_slot;  /* int32 [T] */
  size_t off;         /* int32 [E_l+1] */
  size_t sub_off;     /* int32 [4][E_l][9]: chunk offsets for K = 1,2,4,8:
                         entry q of (K option, expert) is the first slot of
                         chunk q, entry K the expert's end */
  size_t row_off;     /* int32 [4][E_l+S][9]: the row map of A, Hbuf and O
                         for K = 1,2,4,8: entry q < K of (K option, segment)
                         is the first row of chunk q of that segment (local
                         experts, then shared experts).  The (segment,
                         chunk) pairs follow each other in segment-major
                         order, each rounded up to a multiple of 32 rows, so
                         every one starts on a 32-row group; within one, rows
                         follow the slots (local experts) or the tokens
                         (shared experts).  Entries q >= K are 0. */
  size_t cnt_rank;    /* int32 [E_l][R] */
  size_t uniq;        /* int32 [R] */
  size_t stats;       /* int32 [16]: X, X_local, X_in, U_local, U_in, bad ids (0-5);
                         gate candidates (8); GEMM tiles of the layer at
                         K = 1, 2, 4, 8 chunks (10-13), written by the table
                         builder for the cost model (section 3.2, Eq 14) */
  size_t plan;        /* moe_plan of the last megakernel launch */
  size_t err;         /* int32 device error word */
  size_t A;           /* bf16 [X_max + 256 E_l + 256][H] (X_max = T*min(k, E_l)):
                         dispatched rows at the rows of the row map of the
                         launch's chunk count, group-tiled: row r, column j
                         at element ((r/32)*(H/32) + j/32)*1024 + (r%32)*32 + j%32 */
  size_t Hbuf;        /* bf16 [rows of A + S*(Tr + 256)][F]: SiLU(gate)*up,
                         the same row map, group-tiled like A (F in place of H) */
  size_t O;           /* bf16 [rows of Hbuf][H]: expert outputs, the same row
                         map, row-major */
} moe_ws_layout;

/* Creates a handle.  cfg (host) is copied; calib (host) may be NULL for the
 * built-in MI355X calibration.  Validates the shape; does not touch the GPU
 * beyond querying the current device's CU count.  *out receives the handle. */
moe_status moe_init(const moe_config* cfg, const moe_calib* calib, moe_handle** out);

/* Releases the handle (host memory only).  NULL is accepted. */
moe_status moe_destroy(moe_handle* h);

/* Thread-local text of the last error returned on this thread ("" if none). */
const char* moe_last_error(void);

/* Replaces the calibration table (host struct, copied; validated against N).
 * The table lives in the workspace: if one is bound it is updated with a
 * synchronous copy, so call this between launches, not while one runs. */
moe_status moe_set_calib(moe_handle* h, const moe_calib* calib);
moe_status moe_get_calib(const moe_handle* h, moe_calib* out);

/* Time limit of every device-side wait of the megakernel (a wait for
 * dispatched rows, finished GEMM tiles or a finished chunk).  When a wait
 * exceeds it the workgroup latches MOE_ERR_TIMEOUT, raises an abort word that
 * makes every other wait give up, and the launch drains and exits.
 * inject_stall != 0 is a test hook that makes every wait target unreachable,
 * so the next megakernel launch exercises this path and exits after ~ms.
 * Default: 2000 ms, no injection. */
moe_status moe_set_timeout_ms(moe_handle* h, double ms, int32_t inject_stall);

/* Test hook for section 4's claim that dynamic claiming tolerates CUs that
 * run at different speeds: with max_sleeps > 0, every workgroup of the
 * megakernel waits a pseudo-random 0..max_sleeps times 64 cycles before
 * taking its arrival ticket and before each GEMM tile, and every wavefront
 * before each dispatch and combine unit it claims.  The counts are drawn
 * from (seed, workgroup, wavefront, event).  Results must not change.
 * max_sleeps in [0, 4096]; 0 (the default) turns it off. */
moe_status moe_set_jitter(moe_handle* h, uint32_t seed, int32_t max_sleeps);

/* Timeline trace of the megakernel (a measurement aid for the schedule of
 * sections 3-4: worker roles, tile waits, movement phases).  buf is caller-
 * owned device memory of `bytes` bytes, or NULL to turn tracing off.  Each
 * later moe_forward in a non-serial mode writes, per wavefront of the launch
 * (S = n_workers * 8 wavefronts, segment b * 8 + w for wavefront w of
 * workgroup b), up to R records into that wavefront's own segment:
 *   bytes 0-63: int32 header: magic 0x31435254, S, R, the int64 word offset
 *     of segment 0
 *   bytes 64..: int32 record count of each segment (S of them), padded to
 *     a multiple of 64 bytes
 *   then S segments of R records of 32 bytes:
 *     int64 word 0: kind | ticket << 8 | xcd << 20 | id << 32
 *     int64 words 1-3: times t0, t1, t2 from the 100 MHz device clock
 * (ticket: the recording workgroup's arrival ticket, which fixes its role:
 * tickets below the plan's c are movement workers; xcd: the XCD it runs on)
 * kind 1 workgroup (id 1 = movement worker): entry, plan + schedule built, exit
 * kind 2 compute tile (id = tile code: stage << 24 | XCD class << 21 |
 *        index): claimed, inputs ready, finished
 * kind 3 dispatch by one movement worker: start, end
 * kind 4 combine unit of one wavefront (id = unit | wave << 24): claimed,
 *        inputs ready (its GEMM1 row tiles done), end
 * kind 5 dispatch unit of one wavefront (id = unit | wave << 24): start,
 *        rows stored and drained, readiness counted
 * R = (bytes - header and counts) / 32 / S; records past R are dropped.  A
 * wavefront appends with a counter of its own (no global atomics).  The
 * counts and header are written at the end of the launch.  The layout of a
 * trace follows the handle's current plan; it changes nothing else.
 * Errors: MOE_ERR_INVALID_ARG for a non-NULL buf too small for one record per
 * wavefront. */
moe_status moe_set_trace(moe_handle* h, void* buf, int64_t bytes);

/* Workspace size in bytes and its region offsets (host out-parameters). */
moe_status moe_workspace_size(const moe_handle* h, size_t* bytes);
moe_status moe_workspace_layout(const moe_handle* h, moe_ws_layout* out);

/* Binds a caller-owned device workspace of at least moe_workspace_size bytes,
 * 256-byte aligned, and initialises its control words on `stream`.  The
 * workspace must stay alive and unused by others while the handle uses it. */
moe_status moe_set_workspace(moe_handle* h, void* ws, size_t bytes, void* stream);

/* Size of the packed expert weights: (E_l + S) * (R(2F) * H + R(H) * F) * 2
 * bytes, R(n) = n rounded up to a multiple of 256 (the operand slabs of the
 * GEMM tiles are padded to 256 rows). */
moe_status moe_packed_weights_size(const moe_handle* h, size_t* bytes);

/* Packs the expert weights into the GEMM operand layout (not part of the
 * layer; done once): each matrix is transposed to k-contiguous rows and
 * stored as 256-row slabs, one 256 x 32 block per 32-deep k-step, so that
 * the GEMM tiles stream whole blocks.  The layout is internal to the
 * library.  w1, w3: bf16 [E_l][H][F] (gate, up), w2: bf16
 * [E_l][F][H] (down); ws1, ws3, ws2 the same for the S shared experts (NULL
 * when S = 0).  packed: device buffer of moe_packed_weights_size bytes. */
moe_status moe_pack_weights(moe_handle* h, const uint16_t* w1, const uint16_t* w3,
                            const uint16_t* w2, const uint16_t* ws1, const uint16_t* ws3,
                            const uint16_t* ws2, void* packed, void* stream);

/* Top-k routing (the routing that precedes the layer, section 4) followed by
 * moe_build_tables.  x: bf16 [T][H] (rank r's rows at r*Tr); wg: bf16 [H][E];
 * logit_bias: fp32 [E] added to the logits, or NULL.  Logits are accumulated
 * in fp32 over ascending h (one accumulator per (token, expert)); the top_k
 * largest logits are selected (ties -> smaller expert id), written in
 * descending order to topk_idx int32 [T][k]; topk_w fp32 [T][k] receives the
 * selected softmax probabilities divided by their sum.  top_k must equal the
 * configured k. */
moe_status moe_route(moe_handle* h, const uint16_t* x, const uint16_t* wg,
                     const float* logit_bias, int32_t top_k, int32_t* topk_idx,
                     float* topk_w, void* stream);

/* Size of the device scratch of moe_route_topk_static: 96 MiB. */
#define MOE_ROUTE_STATIC_SCRATCH_BYTES (96u << 20)

/* The top-k routing of moe_route (gate logits, softmax, top-k,
 * renormalisation; the same kernels and the same results) without a handle
 * and without allocating anything, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation.  It builds no routing tables (moe_build_tables does).
 * x: bf16 [T][H], wg: bf16 [H][E], logit_bias: fp32 [E] or NULL; writes
 * topk_idx int32 [T][top_k] and topk_w fp32 [T][top_k] as moe_route does.
 * The gate's scratch (its intermediate logits, norms and candidate chains,
 * about E*H*2 + 16*T*E + 16*T bytes) lives in a static device array of
 * MOE_ROUTE_STATIC_SCRATCH_BYTES that each GPU the library runs on holds
 * until the process ends; larger problems are refused with
 * MOE_ERR_UNSUPPORTED (nothing is launched).  Every call on a GPU shares that
 * GPU's array and leaves its contents behind: calls that overlap on one GPU
 * (other streams, other threads) race, so serialise them.  H must be a
 * multiple of 64 in [64, 16384], E in [1, 512], top_k in [1, min(E, 8)]. */
moe_status moe_route_topk_static(int32_t T, int32_t H, int32_t E, int32_t top_k, const uint16_t* x,
                                 const uint16_t* wg, const float* logit_bias, int32_t* topk_idx, float* topk_w,
                                 void* stream);

/* Builds the routing tables of this GPU's share from topk_idx int32 [T][k]
 * (section 3.1 descriptors and the dispatch permutation): per-(expert, rank)
 * counts, unique-token counts, expert offsets, the slot of each local pair
 * (slots ordered by local expert, then token), its inverse, each token's
 * first slot and the chunk offsets for K = 1, 2, 4, 8.  Ids outside [0, E) or
 * repeated within a row latch MOE_ERR_ROUTING and are treated as non-local. */
moe_status moe_build_tables(moe_handle* h, const int32_t* topk_idx, void* stream);

/* The MoE layer (section 2.1 stages 1-5) on the tables built from topk_idx.
 * x: bf16 [T][H] staging regions; topk_idx/topk_w: the routing result
 * (topk_idx must be the array the current tables were built from: checked by
 * address); packed: from moe_pack_weights; y: bf16 [T][H] output staging
 * regions, y[g] = sum over local j of topk_w[g,j] * FFN(x[g]) (+ the shared
 * experts for rank-0 tokens), 0 for tokens with no local expert.
 * mode: a moe_mode.  forced: host plan overriding the cost model (c, K,
 * n_steal, final_all) in the megakernel modes, or NULL.
 * The megakernel modes launch one persistent kernel of n_workers workgroups
 * that wait on each other, as an ordinary launch on `stream`: all of them
 * must be resident at once (the first call checks that the GPU holds them:
 * else MOE_ERR_UNSUPPORTED), and work on other streams that holds CUs while
 * it runs can keep workers from starting; the waiting ones then stop at the
 * timeout (moe_set_timeout_ms) with MOE_ERR_TIMEOUT. */
moe_status moe_forward(moe_handle* h, const uint16_t* x, const int32_t* topk_idx,
                       const float* topk_w, const void* packed, uint16_t* y,
                       int32_t mode, const moe_plan* forced, void* stream);

#define MOE_STACK_MAX 12

/* Several MoE layers in one persistent megakernel launch (a stack of
 * independent layers that share the tokens x but not their outputs, as the
 * layers of one GPU's expert-parallel share are when each takes its own
 * routing of the same batch).  layers[l]: the handle of layer l (each with its
 * own workspace, tables built from topk_idx[l], and n_workers equal to layer
 * 0's); packed[l], topk_idx[l], topk_w[l], y[l]: as in moe_forward for that
 * layer (host arrays of device pointers).  Each layer's plan comes from its
 * own prologue (section 3.3), or is `forced` (host, the same for every layer).
 * A workgroup moves on to layer l + 1 as soon as it finds no more work to
 * claim in layer l (section 4's dynamic claiming, across layers), so layer
 * l + 1's dispatch and first GEMM tiles overlap layer l's last tiles and its
 * combine; in every layer but the last, the final combine is left to that
 * layer's movement workers while the compute workers go on to the next
 * layer.  In dynamic mode those movement workers first claim layer l + 1's
 * dispatch units, beside layer l's GEMMs, when layer l + 1's prologue will
 * take a plan known before it runs (forced, or stored with its tables under
 * the current calibration).  Results are those of moe_forward on each layer,
 * bit for bit.
 * mode: MOE_MODE_DYNAMIC or MOE_MODE_STATIC.  1 <= n_layers <= MOE_STACK_MAX,
 * no handle twice.  The timeline trace is not recorded in a stacked launch.
 * Errors: as moe_forward, per layer (device errors latch in each layer's
 * error word). */
moe_status moe_forward_stack(moe_handle* const* layers, int32_t n_layers, const uint16_t* x,
                             const int32_t* const* topk_idx, const float* const* topk_w, const void* const* packed,
                             uint16_t* const* y, int32_t mode, const moe_plan* forced, void* stream);

/* Calibration of the cost model's hardware curves (BW(c), TFLOPS(N-c),
 * eff_chunk(K); Fig 4a/b, Fig 7a): runs the selected stages of the layer as
 * separate kernels on n_workers workgroups.  stages: bit 0 dispatch, bit 1
 * GEMM0 + SiLU*up, bit 2 GEMM1, bit 3 combine; the GEMMs use the tiling of K
 * chunks.  A stage reads what the earlier stages wrote, so a partial mask is
 * meant for timing (after a full run), not for producing y.  Same arguments
 * and table requirement as moe_forward. */
moe_status moe_run_stages(moe_handle* h, const uint16_t* x, const int32_t* topk_idx,
                          const float* topk_w, const void* packed, uint16_t* y,
                          int32_t stages, int32_t n_workers, int32_t K, void* stream);

/* Copies the plan of the last megakernel launch to *out (host).  Synchronises
 * the stream. */
moe_status moe_get_plan(moe_handle* h, moe_plan* out, void* stream);

/* Reads and clears the device error word; synchronises the stream. */
moe_status moe_sync_status(moe_handle* h, void* stream);

/* The cost model alone, on the host, for given routing volumes (fp64, same
 * operation order as the in-kernel prologue).  n_tiles[j]: GEMM tiles at
 * k_chunks[j]. */
moe_status moe_plan_host(const moe_handle* h, double w_comp, double w_dispatch,
                         double w_combine, const int64_t* n_tiles, moe_plan* out);

/* Tile geometry of the grouped GEMM for this shape: rows per tile (bm), GEMM0
 * tiles per row tile (nt0: column tiles over 2F) and GEMM1 tiles per row tile
 * (nt1: column tiles over H times the split-K factor of GEMM1). */
moe_status moe_tile_geometry(const moe_handle* h, int32_t* bm, int32_t* nt0, int32_t* nt1);

#ifdef __cplusplus
}
#endif
#endif
