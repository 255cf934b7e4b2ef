// Kernel argument blocks and launch prototypes shared by the host API and
// the kernels of the MoE-layer library.
#pragma once

#include "common.h"

namespace moe {

struct GateArgs {
  const uint16_t* x;   // [T][H] bf16
  const uint16_t* wg;  // [H][E] bf16
  const float* bias;   // [E] or NULL
  int32_t* topk_idx;
  float* topk_w;
  uint16_t* wgt;       // [E][H] bf16: Wg transposed (workspace)
  float* lt;           // [T][E] approximate logits without bias (workspace)
  float* xn;           // [T] ||x_g||_2 (workspace)
  float* wn;           // [E] ||w_e||_2 (workspace)
  int32_t* ch_g;       // [T * E] chain list: token of each chain (workspace)
  int32_t* ch_e;       // [T * E] expert of each chain
  float* ch_l;         // [T * E] defined logit of each chain
  int32_t* tok_base;   // [T] first chain of each token
  int32_t* tok_n;      // [T] chains of each token
  int32_t* stats;
  float bound;         // |L - L~| <= bound * ||x|| * ||w|| (plus rounding of the bias add)
  int T, H, E, k;
};

struct TableArgs {
  const int32_t* topk_idx;
  int32_t* slot;
  int32_t* inv;
  int32_t* first_slot;
  int32_t* off;
  int32_t* sub_off;
  int32_t* row_off;    // [KOPT][E_l + S][SUBW] first A / Hbuf / O row of each (segment, chunk)
  int32_t* cnt_rank;
  int32_t* uniq;
  int32_t* stats;
  int32_t* blk_cnt;
  int32_t* blk_off;
  int32_t* blk_bad;    // [nblk] tokens with an invalid or repeated id, per table block
  int32_t* rbnd;       // [E_l][R + 1] first slot of each expert at or after each rank boundary
  int32_t* err;
  int T, Tr, R, k, E, e0, El, nblk;
  int S, tiles_per_row_tile;  // shared experts; GEMM0 + GEMM1 tiles of one row tile (the cost model's tile counts)
};

// One source matrix [rows][cols] per segment, written transposed into a
// slab-tiled [R][rows] destination (R = cols, or 2 * cols interleaved).
struct PackArgs {
  const uint16_t* src;
  uint16_t* dst;
  int rows, cols;
  long long seg_stride;
  int interleave, which;
};
// Zeroes rows [R, slab_rows(R)) of every segment's slab-tiled [R][K] matrix.
struct PadArgs {
  uint16_t* dst;
  int nseg, R, K;
  long long seg_stride;
};

// Calibration table as the kernels read it (copied into the workspace).
struct DevCalib {
  int32_t n_c;
  int32_t c[MOE_CALIB_MAX_C];
  double bw[MOE_CALIB_MAX_C];
  double fl[MOE_CALIB_MAX_C];
  int32_t n_k;
  int32_t kk[MOE_CALIB_MAX_K];
  double eff[MOE_CALIB_MAX_K];
  double alpha;
  int32_t literal;
  int32_t static_c;
  double bw_all;  // > 0: the exposed tail moves at this rate (all N workers)
  int32_t steal_window;  // MOE_WINDOW_*: the movement volume of the Eq 11 window
  int32_t steal_ceil;    // Eq 14's share rounded up (1) or down (0)
};

// Schedule of one launch for chunk count K (section 4, the chunk-pipeline DAG
// order): segment seg < E_l is local expert seg, seg >= E_l shared expert
// seg - E_l.  Queue order: chunk, then phase (GEMM0 tiles, then GEMM1 tiles),
// then segment; inside a group the row tile runs fastest (GEMM1: the split
// runs fastest, then the row tile).  Everything from K on depends only on the
// routing tables and the handle, so the routing's last kernel
// (sched_build_kernel) stores it once per K option as an image that a
// launch's prologue copies into LDS once its plan has picked K; the plan
// fields come first and are not part of the image.
struct Sched {
  int c, n_steal, final_all;  // the plan
  int disp0;                  // dispatch units [0, disp0) are owned statically (megakernel)
  int K, nseg, G;             // chunks, segments, groups = K*2*nseg
  int n_comp, n_disp, n_comb;
  int bnd[MAX_K + 1];         // chunk token boundaries ceil(q*T/K)
  // per (chunk q, segment) at index q*nseg + seg
  int rows[MAX_K * MAX_SEG];
  int row0[MAX_K * MAX_SEG];   // first row in Hbuf / O (and in A for local experts), a 32-row group boundary
  int sbase[MAX_K * MAX_SEG];  // first slot (local expert) or token (shared expert) of the segment
  int arow0[MAX_K * MAX_SEG];  // first row of the GEMM0 A operand (A row or token)
  int mb[MAX_K * MAX_SEG];     // first row-tile id (counter index)
  int lvl[MAX_K][NLVL + 1];    // row tiles of chunk q at readiness level <= L
  int gstart[MAX_K * 2 * MAX_SEG + 1];
  int ncls[2 * MAX_K][NXCD];   // tiles of stage (chunk, phase) in slab class x
};
constexpr int SCHED_WORDS = (int)(sizeof(Sched) / 4);  // int32 words of a stored image slot

// The cost model's plan for the tables the schedule images were built from,
// evaluated by sched_build_kernel with the calibration of generation `gen`
// (it follows the images in the workspace).
struct StoredPlan {
  moe_plan p;
  uint32_t gen, pad;
};
constexpr int SCHED_IMG0 = 4;                          // first word of the image (K)

struct FwdArgs {
  // shape
  int T, Tr, R, H, F, k, El, S, e0, N;
  int nt0, nt1;   // column tiles of GEMM0 (over 2F) and GEMM1 (over H)
  int nsplit;     // split-K factor of GEMM1 (1, 2, 4 or 8)
  int dt, ct;     // tokens per dispatch unit (<= DT) and per combine unit (<= CT)
  int move_steal; // compute workers copy dispatch units while their rows are not
                  // ready (dynamic mode; the static split keeps its roles fixed)
  int xmax;       // routed pairs at most (T * min(k, E_l))
  int mt_max;     // capacity of the per-row-tile counters
  int ctl_words;  // int32 words per control set
  int qx, qxs;    // word offsets of the [2 MAX_K][NXCD] tile queue heads (megakernel, serial GEMMs)
  uint32_t calib_gen;  // generation of the calibration table (a StoredPlan of another one is stale)
  // inputs / output
  const uint16_t* x;
  const int32_t* topk_idx;
  const float* topk_w;
  const uint16_t* w13;  // packed [E_l+S] x slab-tiled [2F][H] (gate/up rows interleaved in groups of 32)
  const uint16_t* w2t;  // packed [E_l+S] x slab-tiled [H][F]
  uint16_t* y;
  // routing tables
  const int32_t* slot;
  const int32_t* sub_off;
  const int32_t* row_off;  // [KOPT][E_l + S][SUBW] first row of each (segment, chunk) in A / Hbuf / O
  const int32_t* sched;    // [KOPT][SCHED_WORDS] schedule images (written by sched_build_kernel), K = 1, 2, 4, 8
  const int32_t* stats;
  // intermediate buffers
  uint16_t* A;
  uint16_t* Hb;
  uint16_t* O;
  float* part;    // split-K partials of GEMM1, fp32 [nsplit][prow][H] (nsplit > 1)
  size_t prow;    // rows per split in part (the row capacity of Hbuf and O)
  long long* trace;  // timeline buffer (NULL: off), see moe_set_trace
  int trace_cap;     // records per wavefront segment
  int trace_rec0;    // int64 word offset of the first segment
  // control
  int32_t* ctl;       // this launch's control set
  int32_t* ctl_next;  // cleared for the next launch
  int32_t* err;
  moe_plan* plan_out;
  const DevCalib* calib;
  int mode;           // MOE_MODE_DYNAMIC or MOE_MODE_STATIC
  int forced;
  moe_plan fplan;
  long long timeout_ticks;  // per wait, 100 MHz ticks
  int inject_stall;         // test hook: every wait targets an unreachable value
  uint32_t jitter_seed;     // test hook: seeded random delays (moe_set_jitter)
  int jitter_max;           //   at most this many 64-cycle sleeps per event; 0 = off
  int serial_K;             // chunk tiling used by the separate-kernel GEMMs
  int static_disp;          // megakernel: the first round of dispatch units is owned by arrival ticket
  int stack_next;           // stacked launch: another layer follows, so compute workers go on to it
                            // instead of joining this layer's final combine (its movement workers do it)
};

// Layers of one stacked megakernel launch, their argument blocks by value
// (kernel arguments: read by scalar loads, like a single launch's).
constexpr int STACK_MAX = MOE_STACK_MAX;
struct StackArgs {
  int n;
  FwdArgs layer[STACK_MAX];
};
static_assert(sizeof(StackArgs) <= 4096, "the stacked launch's arguments fit the kernel argument segment");

// ---- cost model (sections 3.1-3.3) ------------------------------------------
// Evaluates T_total(c, K) of Eq 15 over the calibrated (c, K) grid, takes the
// first strict minimum (c ascending, then K ascending; Eq 16), then the steal
// count of Eq 11-14 at (c*, K*).  fp64, no contraction; the host entry point
// and the megakernel prologue run this same function.
__host__ __device__ inline double cm_t_total(const DevCalib& cb, int ci, int ki, double w_comp,
                                             double w_disp, double w_comb) {
#pragma clang fp contract(off)
  double bw = cb.bw[ci];
  double fl = cb.fl[ci];
  double K = (double)cb.kk[ki];
  double t_comp = w_comp / (fl * cb.eff[ki]);                // Eq 9 (Eq 4 at K = 1)
  double t_comm = (w_disp + w_comb) / bw;                    // Eq 5
  // Eq 10 (Eq 6 at K = 1); the last chunk's combine runs on all N workers
  // (section 4), at the calibrated all-worker rate when one is given
  double bw_tail = cb.bw_all > 0.0 ? cb.bw_all : bw;
  double t_tail = ((1.0 - cb.alpha) * w_comb) / (bw_tail * K);
  double s = t_comp + t_tail;
  return s > t_comm ? s : t_comm;                            // Eq 15 (Eq 7 at K = 1)
}

// The steal count of Eq 11-14 at the chosen (c*, K*) = grid point (bc, bk)
// with T_total = best, and the plan.
__host__ __device__ inline void cm_finish(const DevCalib& cb, int N, double w_comp, double w_disp, double w_comb,
                                          const long long* n_tiles_by_k, int bc, int bk, double best,
                                          moe_plan* out) {
#pragma clang fp contract(off)
  // Eq 11 over the window the movement workers have while the GEMMs run
  // (W_comm is not defined there): the whole movement volume of Eq 5
  // (MOE_WINDOW_PLAIN); less the last chunk's combine, which runs on all N
  // workers afterwards (MOE_WINDOW_LAST_COMBINE); less also the first chunk's
  // dispatch when all workers copy it before any GEMM tile starts (movement
  // stealing, MOE_WINDOW_MOVE_STEAL)
  const double kd = (double)cb.kk[bk];
  double w_win = w_disp + w_comb;
  if (cb.steal_window == MOE_WINDOW_MOVE_STEAL) w_win = ((w_disp + w_comb) * (kd - 1.0)) / kd;
  else if (cb.steal_window == MOE_WINDOW_LAST_COMBINE) w_win = w_disp + (w_comb * (kd - 1.0)) / kd;
  double t_comm = w_win / cb.bw[bc];                         // Eq 11
  double w_partial = t_comm * cb.fl[bc];                     // Eq 12
  double w_steal = w_comp - w_partial;                       // Eq 13
  if (w_steal < 0.0) w_steal = 0.0;
  long long nt = n_tiles_by_k[bk];
  int n_steal = 0;
  if (nt > 0 && w_comp > 0.0) {
    double w_tile = w_comp / (double)nt;
    // Eq 14 gives a share, not a count: whole tiles, or the share rounded up
    // (a movement worker's claims stop anyway once the queue is empty)
    const double share = w_steal / ((double)N * w_tile);    // Eq 14
    n_steal = (int)(cb.steal_ceil ? ceil(share) : floor(share));
  }
  out->c = cb.c[bc];
  out->K = cb.kk[bk];
  out->n_steal = n_steal;
  out->final_all = 1;
  out->t_pred_s = best;
}

// Eq 16: argmin of T_total over the grid, c ascending then K ascending, the
// first strict minimum winning; then the steal count.  (The megakernel's
// prologue evaluates the grid points in parallel and scans them in the same
// order, with the same bits.)
__host__ __device__ inline void cost_model(const DevCalib& cb, int N, double w_comp, double w_disp,
                                           double w_comb, const long long* n_tiles_by_k,
                                           moe_plan* out) {
#pragma clang fp contract(off)
  int bc = 0, bk = 0;
  double best = cm_t_total(cb, 0, 0, w_comp, w_disp, w_comb);
  for (int ci = 0; ci < cb.n_c; ++ci)
    for (int ki = 0; ki < cb.n_k; ++ki) {
      double t = cm_t_total(cb, ci, ki, w_comp, w_disp, w_comb);
      if (t < best) { best = t; bc = ci; bk = ki; }
    }
  cm_finish(cb, N, w_comp, w_disp, w_comb, n_tiles_by_k, bc, bk, best, out);
}

// Volumes of section 3.1 from the routing stats.  With `literal` the moved
// bytes are Eq 2-3 as printed (remote rows only); otherwise every moved row
// counts, since on one GPU rank 0's rows also pass through the movement
// workers.  Shared-expert rows are compute-only work.
__host__ __device__ inline void cm_volumes(const int32_t* stats, int H, int F, int shared_rows,
                                           int literal, double* w_comp, double* w_disp,
                                           double* w_comb) {
#pragma clang fp contract(off)
  double B = 2.0 * (double)H;
  double X = (double)stats[ST_X];
  *w_comp = (((X + (double)shared_rows) * 6.0) * (double)H) * (double)F;   // Eq 1
  if (literal) {
    *w_disp = (double)stats[ST_UIN] * B;                                   // Eq 2
    *w_comb = (double)stats[ST_XIN] * B;                                   // Eq 3
  } else {
    *w_disp = ((double)stats[ST_ULOCAL] + (double)stats[ST_UIN]) * B;
    *w_comb = X * B;
  }
}

constexpr int GATE_WAVES = 4;  // wavefronts per workgroup of gate_mfma_kernel (each sums a quarter of H)

// ---- launch prototypes ---------------------------------------------------------
__global__ void gate_prep_kernel(GateArgs a);
__global__ void gate_mfma_kernel(GateArgs a);
template <int GT_M, int EPL>
__global__ void gate_tile_kernel(GateArgs a);  // E > 32; GT_M tokens per workgroup (64 or 128),
                                               // EPL >= E / 16 experts per lane in the candidate pass
__global__ void gate_chain_kernel(GateArgs a);
template <int CX, int NP>
__global__ void gate_chain_staged_kernel(GateArgs a);  // E <= 128, CX tokens per range, NP stages
constexpr int GATE_CHAIN_STAGED_W = 512;               // chains per workgroup of gate_chain_staged_kernel
template <int GT_M>
__global__ void gate_tile2_kernel(GateArgs a);  // 32 < E <= 128; GT_M tokens per workgroup (64 or 128)
template <int EPL, bool COUNT>
__global__ void gate_final_kernel(GateArgs a, TableArgs t);  // EPL >= E / 16 experts per lane; COUNT: also
                                                             // tab_count_kernel's step on the chosen ids
__global__ void tab_count_kernel(TableArgs a);
__global__ void tab_scan_kernel(TableArgs a);
__global__ void tab_perm_kernel(TableArgs a);
__global__ void tab_finalize_kernel(TableArgs a);
constexpr int TAB_SCAN_THREADS = 1024;  // one workgroup of tab_scan_kernel
__global__ void zero_i32_kernel(int* p, int n);
__global__ void pack_transpose_kernel(PackArgs a);
__global__ void pack_pad_kernel(PadArgs a);
__global__ void moe_megakernel(FwdArgs a);
__global__ void moe_megakernel_stack(StackArgs st);
__global__ void sched_build_kernel(FwdArgs a);  // one workgroup per K option
__global__ void serial_dispatch_kernel(FwdArgs a);
__global__ void serial_gemm0_kernel(FwdArgs a);
__global__ void serial_gemm1_kernel(FwdArgs a);
__global__ void serial_combine_kernel(FwdArgs a);

}  // namespace moe
