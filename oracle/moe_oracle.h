/*
 * CPU oracle for one GPU's share of an expert-parallel MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg may call this library.  It shares no code, header, table or
 * helper with the HIP path, and the HIP path never calls it.
 *
 * Plain, single-threaded C.  Each function follows one stage of the layer as
 * the paper defines it (section 2.1 and Fig 3: dispatch, GEMM0 = gate+up
 * projection, SiLU followed by an element-wise product, GEMM1 = down
 * projection, weighted-sum combine), the workload volumes of section 3.1
 * (Eq 1-3) and the cost model of sections 3.1-3.3 (Eq 4-16).
 *
 * Precision.  Routing decides integers (expert ids), so its logits are taken
 * in fp32, the kernel's precision, in one pinned order (ascending hidden index,
 * one accumulator).  Each product of two bf16 values is exact in fp32, so a
 * fused or unfused multiply-add gives the same sum.  Softmax weights, the
 * expert FFN and the combine are computed in fp64 from the bf16 inputs, with
 * no intermediate rounding: that is the exact layer the bf16/fp32 GPU path
 * approximates.  The cost model is fp64 with no contraction, in the operation
 * order written in its comments.
 *
 * bf16 tensors are passed as raw uint16 bit patterns.
 *
 * Parity pins (what checks this oracle against something other than itself)
 * are in tests/test_oracle_pins.py; every function here is pinned.
 */
#ifndef MOE_ORACLE_H
#define MOE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Gate logits (routing happens before the MoE layer, section 4: the routing
 * result is the megakernel's input).  logits[g*E+e] = sum_h x[g,h]*wg[h,e]
 * accumulated in fp32 for h = 0,1,...,H-1 from 0.0f, then + bias[e] (bias may
 * be NULL).  x: [T,H], wg: [H,E] (row-major bf16 bits), logits: [T,E]. */
void orc_gate_logits(const uint16_t* x, const uint16_t* wg, const float* bias,
                     int T, int H, int E, float* logits);

/* Softmax over all E logits (fp64), top-k selection on the logits (larger
 * first, equal logits -> smaller expert id), then the selected probabilities
 * divided by their sum.  idx: [T,k] descending; w: [T,k] (fp64). */
void orc_softmax_topk(const float* logits, int T, int E, int k,
                      int32_t* idx, double* w);

/* Routing tables of this GPU's share (section 3.1 and section 4).
 * Local experts are [e0, e0+El); token g belongs to source rank g / Tr.
 * A local pair (g,j) has le = idx[g,j]-e0 in [0,El).  Slots of the
 * expert-contiguous buffer are numbered by (le ascending, g ascending).
 *   cnt_rank[le*R + r] : local pairs of expert le from rank r
 *   uniq[r]            : rank-r tokens with at least one local pair
 *   off[le]            : first slot of expert le; off[El] = number of pairs X
 *   slot[g*k+j]        : slot of pair (g,j), or -1 when not local
 *   inv[s]             : g*k+j of the pair in slot s (s < X)
 *   first_slot[g]      : slot of g's pair with the smallest le, or -1
 * Returns X. */
int orc_route_tables(const int32_t* idx, int T, int k, int R, int Tr, int e0, int El,
                     int32_t* cnt_rank, int32_t* uniq, int32_t* off, int32_t* slot,
                     int32_t* inv, int32_t* first_slot);

/* Chunk offsets of the chunk pipeline (section 3.2.1).  Tokens are split into
 * K contiguous chunks, chunk(g) = floor(g*K/T).  sub_off[le*(K+1)+q] is the
 * first slot of expert le holding a token of chunk >= q (q = 0..K). */
void orc_chunk_offsets(const int32_t* inv, const int32_t* off, int T, int k, int El, int K,
                       int32_t* sub_off);

/* Dispatch (section 2.1 stage 1): A[s,:] = x[g,:] for every slot s = 0..X-1,
 * g = inv[s]/k.  A: [X,H] bf16 bits (a pure copy). */
void orc_dispatch(const uint16_t* x, const int32_t* inv, int X, int k, int H, uint16_t* A);

/* One expert's SwiGLU FFN on one row (section 2.1 stages 2-4):
 *   u1 = a.W1, u3 = a.W3 (sum over h), hv = silu(u1)*u3 with
 *   silu(z) = z/(1+exp(-z)), out = hv.W2 (sum over f); fp64 throughout.
 * a: [H], w1,w3: [H,F], w2: [F,H] (bf16 bits), out: [H]. */
void orc_expert_ffn(const uint16_t* a, const uint16_t* w1, const uint16_t* w3,
                    const uint16_t* w2, int H, int F, double* out);

/* Layer output for the listed tokens (section 2.1 stage 5, combine):
 *   y[g] = sum over local j (ascending) of w[g,j] * FFN_{idx[g,j]}(x[g])
 *        + (g in rank 0) * sum_s FFN^shared_s(x[g])
 * and y[g] = 0 for tokens with neither.  w1,w3: [El,H,F], w2: [El,F,H];
 * ws1/ws3/ws2 likewise for S shared experts (may be NULL when S == 0).
 * y: [n_rows, H] fp64, row i for token rows[i]. */
void orc_layer_rows(const uint16_t* x, const int32_t* idx, const double* w,
                    const uint16_t* w1, const uint16_t* w3, const uint16_t* w2,
                    const uint16_t* ws1, const uint16_t* ws3, const uint16_t* ws2,
                    int k, int Tr, int H, int F, int e0, int El, int S,
                    const int64_t* rows, int n_rows, double* y);

/* Number of GEMM tiles of the chunked grouped GEMM for chunk count K, given
 * the row count of every (segment, chunk): rows_seg[seg*K + q].  Each
 * segment's rows are cut into ceil(rows/BM) row tiles; GEMM0 has nt0 column
 * tiles per row tile and GEMM1 nt1. */
int64_t orc_tile_count(const int32_t* rows_seg, int n_seg, int K, int BM, int nt0, int nt1);

/* Cost model (sections 3.1-3.3). */
typedef struct {
  /* hardware input: candidate comm-worker counts c[i] with the calibrated
   * bandwidth BW(c[i]) (bytes/s) and GEMM throughput TFLOPS(N - c[i])
   * (flop/s); chunk counts K[j] with eff_chunk(K[j]); overlap ratio alpha */
  int n_c;
  const int32_t* c;
  const double* bw;
  const double* flops;
  int n_k;
  const int32_t* K;
  const double* eff;
  double alpha;
  int N;                 /* workers available to the megakernel */
  /* software input (routing-derived, section 3.1) */
  double w_comp;         /* Eq 1, flop */
  double w_dispatch;     /* Eq 2, bytes */
  double w_combine;      /* Eq 3, bytes */
  const int64_t* n_tiles; /* GEMM tiles for each K[j] (W_tile = w_comp / n_tiles) */
  /* rate of all N workers moving together (bytes/s); the last chunk's combine
   * runs on every worker (section 4), so when bw_all > 0 the exposed tail of
   * Eq 6/10 moves at bw_all, else at BW(c) as printed */
  double bw_all;
  /* which movement work the window of Eq 11 holds (the paper leaves W_comm
   * undefined there):
   *   0  W_dispatch + W_combine, the volume of Eq 5 (the plain reading);
   *   1  (W_dispatch + W_combine)(K-1)/K: the first chunk's dispatch runs on
   *      all N workers before any GEMM tile starts (compute workers copy the
   *      rows they wait for) and the last chunk's combine runs on all N
   *      workers after the GEMMs (section 4), so neither is left to the
   *      movement workers while the GEMMs run;
   *   2  W_dispatch + W_combine (K-1)/K: only the last chunk's combine is
   *      outside the window. */
  int steal_window;
  /* Eq 14 gives each movement worker a share W_steal / (N W_tile) of tiles;
   * 0 takes its whole part (floor), 1 rounds it up (claims stop anyway once
   * the compute queue is empty) */
  int steal_ceil;
} orc_plan_in;

typedef struct {
  int c;           /* c* */
  int K;           /* K* */
  int n_steal;     /* tiles each comm worker steals (Eq 11-14 at c*, K*) */
  int ci, ki;      /* grid indices of c*, K* */
  double t_total;  /* T_total(c*, K*) */
} orc_plan_out;

/* Evaluates Eq 10, 9 (with Eq 5) and 15 for every (c, K) in the grid, takes
 * the argmin of Eq 16 (c ascending, then K ascending, first strict minimum
 * wins), then n_steal from Eq 11-14 at (c*, K*). */
void orc_plan(const orc_plan_in* in, orc_plan_out* out);

/* T_total(c[ci], K[ki]) of Eq 15 (exposed for the closed-form pins). */
double orc_t_total(const orc_plan_in* in, int ci, int ki);

#ifdef __cplusplus
}
#endif
#endif
