// The MoE layer on one GPU's share (paper section 2.1, Fig 3), run either as
// one persistent megakernel with movement and compute workers (sections 3-4)
// or as four separate kernels (the serial baseline, "w/o S+T" of section 5.6).
//
// Data layout in HBM
//   x    bf16 [T][H]        staging regions: rank r's rows at r*Tr
//   A    bf16 [X+pad][H]    dispatched rows, expert-contiguous (slot order)
//   Hbuf bf16 [X+S*Tr+pad][F]  SiLU(gate)*up per row (shared experts after X)
//   O    bf16 [X+S*Tr+pad][H]  expert outputs per row
//   part fp32 [row tile][col tile][split][256*256]  split-K partials of GEMM1
//   y    bf16 [T][H]        output staging regions
//   w13  bf16 [E_l+S][2F][H] gate/up weights, k-contiguous, 32-col interleave
//   w2t  bf16 [E_l+S][H][F]  down weights, k-contiguous
#include "common.h"
#include "gemm.h"
#include "kernels.h"

namespace moe {

constexpr int NWF = FNTH / WAVE;  // waves per forward workgroup

// ===========================================================================
// Schedule of one launch for chunk count K (built by every workgroup in LDS).
// Segment seg < E_l is local expert seg; seg >= E_l is shared expert seg-E_l.
// Queue order (section 4, chunk-pipeline DAG order): chunk, then phase (GEMM0
// tiles, then GEMM1 tiles), then segment; inside a group the row tile runs
// fastest (GEMM1: the split runs fastest, then the row tile).
// ===========================================================================
struct Sched {
  int K, nseg, G;        // chunks, segments, groups = K*2*nseg
  int n_comp, n_disp, n_comb;
  int c, n_steal, final_all;
  int bnd[MAX_K + 1];    // chunk token boundaries ceil(q*T/K)
  int cstart[MAX_K + 1]; // combine units before chunk q
  int g1need[MAX_K];     // GEMM1 (row, column) tiles of chunk q
  // per (chunk q, segment) at index q*nseg + seg
  int rows[MAX_K * MAX_SEG];
  int row0[MAX_K * MAX_SEG];   // first row in Hbuf / O (and in A for local experts)
  int arow0[MAX_K * MAX_SEG];  // first row of the GEMM0 A operand (A slot or token)
  int mb[MAX_K * MAX_SEG];     // first row-tile id (counter index)
  int gstart[MAX_K * 2 * MAX_SEG + 1];
};

struct Scratch {
  int bc[8];
  long long ntk[KOPT];
  int part[NWF];
  int wsl[NWF][WAVE];    // per wavefront: slots of its unit's (token, j) pairs
  float wwt[NWF][WAVE];  // per wavefront: their weights
};

// block-wide exclusive scan of n ints in LDS (all threads call): each thread
// sums a contiguous run, wavefront shuffles scan the run sums, then the runs
// are rewritten with their offsets
__device__ __forceinline__ void block_exscan(int* v, int n, int* part) {
  const int tid = threadIdx.x;
  const int lane = tid & (WAVE - 1), wave = tid / WAVE;
  const int per = (n + FNTH - 1) / FNTH;
  const int b = tid * per, e = min(n, b + per);
  int mine = 0;
  for (int i = b; i < e; ++i) mine += v[i];
  int x = mine;
#pragma unroll
  for (int d = 1; d < WAVE; d <<= 1) {
    int y = __shfl_up(x, d, WAVE);
    if (lane >= d) x += y;
  }
  if (lane == WAVE - 1) part[wave] = x;
  __syncthreads();
  int run = x - mine;
  for (int w = 0; w < wave; ++w) run += part[w];
  for (int i = b; i < e; ++i) { int t = v[i]; v[i] = run; run += t; }
  __syncthreads();
}

__device__ __forceinline__ void build_sched(const FwdArgs& a, Sched& S, Scratch& W, int K) {
  const int tid = threadIdx.x;
  const int ki = kopt_index(K);
  const int nseg = a.El + a.S;
  const int g1tiles = a.nt1 * a.nsplit;  // GEMM1 tiles per row tile
  if (tid == 0) {
    S.K = K;
    S.nseg = nseg;
    S.G = K * 2 * nseg;
    for (int q = 0; q <= K; ++q) S.bnd[q] = (int)(((long long)q * a.T + K - 1) / K);
    int cs = 0;
    for (int q = 0; q < K; ++q) { S.cstart[q] = cs; cs += ceil_div(S.bnd[q + 1] - S.bnd[q], CT); }
    S.cstart[K] = cs;
    S.n_comb = cs;
    S.n_disp = ceil_div(a.T, DT);
  }
  __syncthreads();
  for (int v = tid; v < K * nseg; v += FNTH) {
    int q = v / nseg, seg = v % nseg;
    int rows, row0, arow0;
    if (seg < a.El) {
      const int* so = a.sub_off + ((size_t)ki * a.El + seg) * SUBW;
      row0 = so[q];
      rows = so[q + 1] - so[q];
      arow0 = row0;
    } else {
      int s = seg - a.El;
      int t0 = S.bnd[q], t1 = min(S.bnd[q + 1], a.Tr);
      rows = max(0, t1 - t0);
      arow0 = t0;
      row0 = a.xmax + s * a.Tr + t0;
    }
    S.rows[v] = rows;
    S.row0[v] = row0;
    S.arow0[v] = arow0;
    S.mb[v] = ceil_div(rows, BM);
  }
  __syncthreads();
  for (int gi = tid; gi < S.G; gi += FNTH) {
    int q = gi / (2 * nseg), ph = (gi / nseg) & 1, seg = gi % nseg;
    S.gstart[gi] = S.mb[q * nseg + seg] * (ph ? g1tiles : a.nt0);
  }
  if (tid == 0) S.gstart[S.G] = 0;
  if (tid < K) {
    int s = 0;
    for (int seg = 0; seg < nseg; ++seg) s += S.mb[tid * nseg + seg] * a.nt1;
    S.g1need[tid] = s;
  }
  __syncthreads();
  block_exscan(S.mb, K * nseg, W.part);
  block_exscan(S.gstart, S.G + 1, W.part);
  if (tid == 0) S.n_comp = S.gstart[S.G];
  __syncthreads();
}

// ===========================================================================
// Movement work, one wavefront per unit (no workgroup barriers, so the eight
// wavefronts of a movement worker overlap their latency chains):
// dispatch copies the rows of DT tokens into their expert-contiguous A slots
// (each row read once, written to every local slot); combine writes the
// weighted sum of the expert outputs of CT tokens into the output staging
// region.
// ===========================================================================
__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / WAVE; }

__device__ __forceinline__ int wave_claim(int* q) {
  int v = 0;
  if (lane_id() == 0) v = fetch_add_relaxed(q, 1);
  return __builtin_amdgcn_readfirstlane(v);
}

__device__ __forceinline__ void dispatch_unit(const FwdArgs& a, const Sched* S, Scratch& W, int u, bool signal) {
  const int lane = lane_id();
  int* sl = W.wsl[wave_id()];
  const int g0 = u * DT;
  const int nt = min(DT, a.T - g0);
  const int k = a.k;
  sl[lane] = lane < nt * k ? a.slot[(size_t)g0 * k + lane] : -1;
  __builtin_amdgcn_wave_barrier();
  const int VPR = a.H >> 3;
  const int total = nt * VPR;
  constexpr int VB = 16;  // 16-byte vectors per lane in flight
  for (int v0 = lane; v0 < total; v0 += VB * WAVE) {
    u32x4_t val[VB];
    int tt[VB], cc[VB];
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = v0 + i * WAVE;
      tt[i] = -1;
      if (v < total) {
        const int t = v / VPR;
        const int c = v - t * VPR;
        bool any = false;
        for (int j = 0; j < k; ++j) any |= (unsigned)sl[t * k + j] < (unsigned)a.xmax;
        if (any) {
          tt[i] = t;
          cc[i] = c;
          val[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.x + (size_t)(g0 + t) * a.H + c * 8));
        }
      }
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      if (tt[i] < 0) continue;
      for (int j = 0; j < k; ++j) {
        const int s = sl[tt[i] * k + j];
        if ((unsigned)s < (unsigned)a.xmax) *reinterpret_cast<u32x4_t*>(a.A + (size_t)s * a.H + cc[i] * 8) = val[i];
      }
    }
  }
  if (signal) {
    // this wavefront's rows are complete and written back before it counts
    // them in the readiness counters of their row tiles
    __builtin_amdgcn_s_waitcnt(0);
    fence_release_agent();
    if (lane < nt * k) {
      const int s = sl[lane];
      const int g = g0 + lane / k;
      const int le = (unsigned)s < (unsigned)a.xmax ? a.topk_idx[(size_t)g * k + (lane % k)] - a.e0 : -1;
      if ((unsigned)le < (unsigned)a.El) {
        const int q = (int)(((long long)g * S->K) / a.T);
        const int id = S->mb[q * S->nseg + le] + (s - S->row0[q * S->nseg + le]) / BM;
        if ((unsigned)id < (unsigned)a.mt_max) fetch_add_relaxed(&a.ctl[CTL_READY + id], 1);
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
}

// One wavefront combines nt <= CT tokens.  Each token has KS = k + S source
// rows in O: its k routed slots (weight w, absent when the expert is not
// local) followed by its S shared-expert rows (weight 1, present for tokens of
// rank 0).  They are summed in that order in fp32.  KS is a template constant
// so that every lane keeps about 16 row vectors in flight.
template <int KS>
__device__ __forceinline__ void combine_body(const FwdArgs& a, const int* sl, const float* wt, int g0, int nt) {
  constexpr int P = KS >= 16 ? 1 : 16 / KS;  // positions per lane per pass
  const int lane = lane_id();
  const int VPR = a.H >> 3;
  const int total = nt * VPR;
  for (int v0 = lane; v0 < total; v0 += P * WAVE) {
    u32x4_t o[P][KS];
    int tt[P], cc[P];
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int v = v0 + i * WAVE;
      tt[i] = v < total ? v / VPR : -1;
      cc[i] = v < total ? v - tt[i] * VPR : 0;
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        const int s = tt[i] >= 0 ? sl[tt[i] * KS + j] : -1;
        if (s >= 0) o[i][j] = *reinterpret_cast<const u32x4_t*>(a.O + (size_t)s * a.H + cc[i] * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < P; ++i) {
      if (tt[i] < 0) continue;
      float acc[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        if (sl[tt[i] * KS + j] < 0) continue;
        const float w = wt[tt[i] * KS + j];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] += w * bf16_lo(o[i][j][q]);
          acc[2 * q + 1] += w * bf16_hi(o[i][j][q]);
        }
      }
      u32x4_t r;
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = pack_bf16x2(acc[2 * q], acc[2 * q + 1]);
      __builtin_nontemporal_store(r, reinterpret_cast<u32x4_t*>(a.y + (size_t)(g0 + tt[i]) * a.H + cc[i] * 8));
    }
  }
}

__device__ __forceinline__ void combine_tokens(const FwdArgs& a, Scratch& W, int g0, int nt) {
  const int lane = lane_id();
  int* sl = W.wsl[wave_id()];
  float* wt = W.wwt[wave_id()];
  const int k = a.k, ks = a.k + a.S;
  // source rows of token g0 + lane / ks, entry lane % ks
  if (lane < nt * ks) {
    const int t = lane / ks, j = lane - t * ks, g = g0 + t;
    int s = -1;
    float w = 1.0f;
    if (j < k) {
      s = a.slot[(size_t)g * k + j];
      w = a.topk_w[(size_t)g * k + j];
      if ((unsigned)s >= (unsigned)a.xmax) s = -1;
    } else if (g < a.Tr) {
      s = a.xmax + (j - k) * a.Tr + g;
    }
    sl[lane] = s;
    wt[lane] = w;
  }
  __builtin_amdgcn_wave_barrier();
  switch (ks) {
#define MOE_COMBINE_CASE(n) case n: combine_body<n>(a, sl, wt, g0, nt); break;
    MOE_COMBINE_CASE(1) MOE_COMBINE_CASE(2) MOE_COMBINE_CASE(3) MOE_COMBINE_CASE(4)
    MOE_COMBINE_CASE(5) MOE_COMBINE_CASE(6) MOE_COMBINE_CASE(7) MOE_COMBINE_CASE(8)
    MOE_COMBINE_CASE(9) MOE_COMBINE_CASE(10) MOE_COMBINE_CASE(11) MOE_COMBINE_CASE(12)
    MOE_COMBINE_CASE(13) MOE_COMBINE_CASE(14) MOE_COMBINE_CASE(15) MOE_COMBINE_CASE(16)
#undef MOE_COMBINE_CASE
    default: break;
  }
  __builtin_amdgcn_wave_barrier();
}

// ===========================================================================
// Compute work: one tile of GEMM0 (+SiLU*up) or one split of a GEMM1 tile.
// ===========================================================================
struct TileRef {
  int q, ph, seg, mt, nt, ks, rows;
};

__device__ __forceinline__ TileRef decode_tile(const FwdArgs& a, const Sched& S, int t) {
  int lo = 0, hi = S.G;  // the group gi with gstart[gi] <= t < gstart[gi+1]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (S.gstart[mid] <= t) lo = mid; else hi = mid;
  }
  TileRef r;
  r.q = lo / (2 * S.nseg);
  r.ph = (lo / S.nseg) & 1;
  r.seg = lo % S.nseg;
  int local = t - S.gstart[lo];
  const int rows = S.rows[r.q * S.nseg + r.seg];
  const int nmt = ceil_div(rows, BM);
  if (r.ph == 0) {
    r.ks = 0;
  } else {
    r.ks = local % a.nsplit;
    local /= a.nsplit;
  }
  r.mt = local % nmt;
  r.nt = local / nmt;
  r.rows = min(BM, rows - r.mt * BM);
  return r;
}

__device__ __forceinline__ void signal_done(int* p) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(p, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Runs the tile; returns true when it completed an output tile (GEMM0 tile,
// or the last-arriving split of a GEMM1 tile, which did the reduction).
// One mainloop instance serves both GEMMs; only the operands and the
// epilogue differ.
__device__ __forceinline__ bool run_gemm(const FwdArgs& a, const Sched& S, Scratch& W, const TileRef& r, int mtile_id,
                                         char* ring) {
  const int qs = r.q * S.nseg + r.seg;
  const size_t orow = (size_t)S.row0[qs] + (size_t)r.mt * BM;
  const int n0 = r.nt * BN;
  const uint16_t* Aop;
  const uint16_t* Bop;
  int ld, b_rows, Kd;
  if (r.ph == 0) {
    const size_t arow = (size_t)S.arow0[qs] + (size_t)r.mt * BM;
    Aop = (r.seg < a.El ? a.A : a.x) + arow * a.H;
    Bop = a.w13 + ((size_t)r.seg * 2 * a.F + n0) * a.H;
    ld = a.H;
    b_rows = 2 * a.F - n0;
    Kd = a.H;
  } else {
    const int kl = a.F / a.nsplit;
    Aop = a.Hb + orow * a.F + (size_t)r.ks * kl;
    Bop = a.w2t + ((size_t)r.seg * a.H + n0) * a.F + (size_t)r.ks * kl;
    ld = a.F;
    b_rows = a.H - n0;
    Kd = kl;
  }
  gemm::Acc acc;
  gemm::zero(acc);
  gemm::mainloop(acc, Aop, ld, r.rows, Bop, ld, b_rows, Kd, ring);
  if (r.ph == 0) {
    gemm::store_silu_mul(acc, a.Hb + orow * a.F + n0 / 2, a.F, r.rows, a.F - n0 / 2);
    return true;
  }
  uint16_t* out = a.O + orow * a.H + n0;
  if (a.nsplit == 1) {
    gemm::store_bf16(acc, out, a.H, r.rows, a.H - n0);
    return true;
  }
  // split-K: publish this split's partial; the last arrival reduces in order
  const size_t tile = (size_t)mtile_id * a.nt1 + r.nt;
  float* parts = a.part + tile * a.nsplit * (size_t)(BM * BN);
  gemm::store_partial(acc, parts + (size_t)r.ks * (BM * BN));
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    W.bc[3] = __hip_atomic_fetch_add(&a.ctl[CTL_READY + 2 * a.mt_max + tile], 1, __ATOMIC_RELEASE,
                                     __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const bool last = W.bc[3] == a.nsplit - 1;
  __syncthreads();
  if (!last) return false;
  if (a.nsplit == 2) gemm::reduce_store<2>(parts, (size_t)(BM * BN), out, a.H, r.rows, a.H - n0);
  else gemm::reduce_store<4>(parts, (size_t)(BM * BN), out, a.H, r.rows, a.H - n0);
  return true;
}

// ===========================================================================
// Prologue: the routing-derived workload and the plan (sections 3.1-3.3),
// computed redundantly by every workgroup from a small read of the stats.
// ===========================================================================
__device__ __forceinline__ void prologue_plan(const FwdArgs& a, Sched& S, Scratch& W) {
  const int tid = threadIdx.x;
  const int nseg = a.El + a.S;
  if (tid < KOPT) W.ntk[tid] = 0;
  __syncthreads();
  // GEMM tiles at each stored chunk option (for W_tile of Eq 14)
  for (int ki = 0; ki < KOPT; ++ki) {
    const int K = kopt_value(ki);
    long long part = 0;
    for (int v = tid; v < K * nseg; v += FNTH) {
      int q = v / nseg, seg = v % nseg;
      int rows;
      if (seg < a.El) {
        const int* so = a.sub_off + ((size_t)ki * a.El + seg) * SUBW;
        rows = so[q + 1] - so[q];
      } else {
        int t0 = (int)(((long long)q * a.T + K - 1) / K);
        int t1 = min((int)(((long long)(q + 1) * a.T + K - 1) / K), a.Tr);
        rows = max(0, t1 - t0);
      }
      part += (long long)ceil_div(rows, BM) * (a.nt0 + a.nt1 * a.nsplit);
    }
    if (part) atomicAdd((unsigned long long*)&W.ntk[ki], (unsigned long long)part);
  }
  __syncthreads();
  if (tid == 0) {
    moe_plan p;
    if (a.forced) {
      p = a.fplan;
    } else if (a.mode == MOE_MODE_STATIC) {
      p.c = a.calib->static_c;
      p.K = 1;
      p.n_steal = 0;
      p.final_all = 0;
      p.t_pred_s = 0.0;
    } else {
      double wc, wd, wb;
      cm_volumes(a.stats, a.H, a.F, a.S * a.Tr, a.calib->literal, &wc, &wd, &wb);
      long long nt_by_k[MOE_CALIB_MAX_K];
      for (int j = 0; j < a.calib->n_k; ++j) nt_by_k[j] = W.ntk[kopt_index(a.calib->kk[j])];
      cost_model(*a.calib, a.N, wc, wd, wb, nt_by_k, &p);
    }
    S.c = p.c;
    S.K = p.K;
    S.n_steal = p.n_steal;
    S.final_all = p.final_all;
    if (blockIdx.x == 0) *a.plan_out = p;
  }
  __syncthreads();
}

// Waits until *p >= target.  Thread 0 polls with relaxed agent-scope loads
// (coherent across XCDs, no cache invalidation: an acquire here would
// invalidate this XCD's L2 on every poll, under the GEMM tiles of the other
// workgroups).  No acquire is needed for the data that follows: producers
// write back their L2 before publishing (release), and no CU reads a
// dispatched row, an Hbuf/O row or a partial before it is published, so no
// stale copy of those lines can sit in the consumer's L1 or L2 (caches are
// invalidated at kernel start).
__device__ __forceinline__ bool wait_geq(const FwdArgs& a, Scratch& W, const int* p, int target) {
  if (a.inject_stall) target += 1 << 30;
  if (threadIdx.x == 0) {
    int ok = 1;
    if (ld_relaxed(p) < target) {
      const uint64_t deadline = now_ticks() + (uint64_t)a.timeout_ticks;
      while (ld_relaxed(p) < target) {
        if (ld_relaxed(&a.ctl[CTL_ABORT])) { ok = 0; break; }
        if (now_ticks() > deadline) {
          st_relaxed(&a.ctl[CTL_ABORT], 1);
          atomicOr(a.err, ERR_TIMEOUT);
          ok = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
    W.bc[2] = ok;
  }
  __syncthreads();
  const int ok = W.bc[2];
  __syncthreads();
  return ok != 0;
}

__device__ __forceinline__ int claim(Scratch& W, int* q) {
  if (threadIdx.x == 0) W.bc[1] = fetch_add_relaxed(q, 1);
  __syncthreads();
  const int r = W.bc[1];
  __syncthreads();
  return r;
}

// returns false when the launch was aborted
__device__ __forceinline__ bool run_compute_tile(const FwdArgs& a, const Sched& S, Scratch& W, int t, char* ring) {
  TileRef r = decode_tile(a, S, t);
  const int id = S.mb[r.q * S.nseg + r.seg] + r.mt;
  if (r.ph == 0) {
    if (r.seg < a.El && !wait_geq(a, W, &a.ctl[CTL_READY + id], r.rows)) return false;
    run_gemm(a, S, W, r, id, ring);
    signal_done(&a.ctl[CTL_READY + a.mt_max + id]);
  } else {
    if (!wait_geq(a, W, &a.ctl[CTL_READY + a.mt_max + id], a.nt0)) return false;
    if (run_gemm(a, S, W, r, id, ring)) signal_done(&a.ctl[CTL_G1DONE + r.q]);
  }
  return true;
}

// wavefront-level wait: lane 0 polls like wait_geq, the others follow
__device__ __forceinline__ bool wave_wait_geq(const FwdArgs& a, const int* p, int target) {
  if (a.inject_stall) target += 1 << 30;
  int ok = 1;
  if (lane_id() == 0 && ld_relaxed(p) < target) {
    const uint64_t deadline = now_ticks() + (uint64_t)a.timeout_ticks;
    while (ld_relaxed(p) < target) {
      if (ld_relaxed(&a.ctl[CTL_ABORT])) { ok = 0; break; }
      if (now_ticks() > deadline) {
        st_relaxed(&a.ctl[CTL_ABORT], 1);
        atomicOr(a.err, ERR_TIMEOUT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  return __builtin_amdgcn_readfirstlane(ok) != 0;
}

// combine units in chunk order, claimed per wavefront; chunk q's units wait
// until every GEMM1 tile of chunk q is done
__device__ __forceinline__ bool combine_loop(const FwdArgs& a, const Sched& S, Scratch& W) {
  for (;;) {
    const int u = wave_claim(&a.ctl[CTL_Q_COMB]);
    if (u >= S.n_comb) return true;
    int q = 0;
    while (q + 1 < S.K && S.cstart[q + 1] <= u) ++q;
    if (!wave_wait_geq(a, &a.ctl[CTL_G1DONE + q], S.g1need[q])) return false;
    const int g0 = S.bnd[q] + (u - S.cstart[q]) * CT;
    combine_tokens(a, W, g0, min(CT, S.bnd[q + 1] - g0));
  }
}

// ===========================================================================
// The persistent megakernel: one workgroup per CU, co-resident (cooperative
// launch).  The first c workgroups to arrive become movement workers.
// ===========================================================================
__global__ void __launch_bounds__(FNTH, 1) moe_megakernel(FwdArgs a) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(1024))) char ring[gemm::RING_BYTES];
  const int tid = threadIdx.x;

  if (blockIdx.x == 0)
    for (int i = tid; i < a.ctl_words; i += FNTH) a.ctl_next[i] = 0;

  prologue_plan(a, S, W);
  build_sched(a, S, W, S.K);

  if (tid == 0) W.bc[0] = fetch_add_relaxed(&a.ctl[CTL_TICKET], 1);
  __syncthreads();
  const bool mover = W.bc[0] < S.c;
  __syncthreads();

  bool ok = true;
  if (mover) {
    // dispatch: every token row, in token (hence chunk) order, per wavefront
    for (;;) {
      const int u = wave_claim(&a.ctl[CTL_Q_DISP]);
      if (u >= S.n_disp) break;
      dispatch_unit(a, &S, W, u, true);
    }
    __syncthreads();
    // bubble stealing: n_steal GEMM tiles right after dispatch (section 3.2.2)
    for (int i = 0; i < S.n_steal && ok; ++i) {
      const int t = claim(W, &a.ctl[CTL_Q_COMP]);
      if (t >= S.n_comp) break;
      ok = run_compute_tile(a, S, W, t, ring);
    }
    if (ok) combine_loop(a, S, W);
  } else {
    for (;;) {
      const int t = claim(W, &a.ctl[CTL_Q_COMP]);
      if (t >= S.n_comp) break;
      if (!run_compute_tile(a, S, W, t, ring)) { ok = false; break; }
    }
    // final combine on every worker (section 4)
    if (ok && S.final_all) combine_loop(a, S, W);
  }
}

// ===========================================================================
// Serial baseline: four kernels, each on every CU, no overlap.
// ===========================================================================
__global__ void __launch_bounds__(FNTH, 1) serial_dispatch_kernel(FwdArgs a) {
  __shared__ Scratch W;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0)
    for (int i = tid; i < a.ctl_words; i += FNTH) a.ctl_next[i] = 0;
  const int n = ceil_div(a.T, DT);
  for (;;) {
    const int u = wave_claim(&a.ctl[CTL_SQ + 0]);
    if (u >= n) break;
    dispatch_unit(a, nullptr, W, u, false);
  }
}

template <int PH>
__device__ __forceinline__ void serial_gemm(const FwdArgs& a, int qslot) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(1024))) char ring[gemm::RING_BYTES];
  build_sched(a, S, W, a.serial_K);
  // the tiles of phase PH in every chunk, in queue order
  int count = 0;
  for (int q = 0; q < S.K; ++q)
    count += S.gstart[(2 * q + PH + 1) * S.nseg] - S.gstart[(2 * q + PH) * S.nseg];
  for (;;) {
    int t = claim(W, &a.ctl[CTL_SQ + 64 * qslot]);
    if (t >= count) break;
    int q = 0;
    for (;; ++q) {
      const int n = S.gstart[(2 * q + PH + 1) * S.nseg] - S.gstart[(2 * q + PH) * S.nseg];
      if (t < n) break;
      t -= n;
    }
    TileRef r = decode_tile(a, S, S.gstart[(2 * q + PH) * S.nseg] + t);
    run_gemm(a, S, W, r, S.mb[r.q * S.nseg + r.seg] + r.mt, ring);
  }
}

__global__ void __launch_bounds__(FNTH, 1) serial_gemm0_kernel(FwdArgs a) { serial_gemm<0>(a, 1); }
__global__ void __launch_bounds__(FNTH, 1) serial_gemm1_kernel(FwdArgs a) { serial_gemm<1>(a, 2); }

__global__ void __launch_bounds__(FNTH, 1) serial_combine_kernel(FwdArgs a) {
  __shared__ Scratch W;
  const int n = ceil_div(a.T, CT);
  for (;;) {
    const int u = wave_claim(&a.ctl[CTL_SQ + 192]);
    if (u >= n) break;
    const int g0 = u * CT;
    combine_tokens(a, W, g0, min(CT, a.T - g0));
  }
}

}  // namespace moe
