// The MoE layer on one GPU's share (paper section 2.1, Fig 3), run either as
// one persistent megakernel with movement and compute workers (sections 3-4)
// or as four separate kernels (the serial baseline of section 5.6, "w/o S+T").
//
// Data layout in HBM
//   x    bf16 [T][H]        staging regions: rank r's rows at r*Tr
//   A    bf16 [X+pad][H]    dispatched rows, expert-contiguous (slot order)
//   Hbuf bf16 [X+S*Tr+pad][F]  SiLU(gate)*up per row (shared experts after X)
//   O    bf16 [X+S*Tr+pad][H]  expert outputs per row
//   y    bf16 [T][H]        output staging regions
//   w13  bf16 [E_l+S][2F][H] gate/up weights, k-contiguous, 32-col interleave
//   w2t  bf16 [E_l+S][H][F]  down weights, k-contiguous
#include "common.h"
#include "kernels.h"

namespace moe {

// ===========================================================================
// Grouped-GEMM tile: C[BM x BN] = A[BM x Kd] * B[BN x Kd]^T on bf16 MFMA
// (v_mfma_f32_32x32x16_bf16), fp32 accumulation.  4 waves in a 2 x 2 grid,
// each wave owns 64 x 128 outputs (2 x 4 MFMA blocks).  A and B stream
// through double-buffered LDS tiles of BK = 64; 16-byte chunks are XOR-swizzled
// by row so the fragment reads are free of bank conflicts.
// EPI 0 (GEMM0): columns come in gate/up 32-column pairs; the epilogue writes
//   bf16(silu(gate) * up), BN/2 columns.
// EPI 1 (GEMM1): the epilogue writes bf16(C), BN columns.
// ===========================================================================
constexpr int GEMM_SMEM = 2 * (BM * BK + BN * BK) * 2;  // bytes (96 KiB)

__device__ __forceinline__ int swz(int row, int chunk) { return row * BK + ((chunk ^ (row & 7)) << 3); }

template <int EPI>
__device__ void gemm_tile(const uint16_t* __restrict__ A, int lda, int a_rows,
                          const uint16_t* __restrict__ B, int ldb, int b_rows, int Kd,
                          uint16_t* __restrict__ out, int ldo, int out_rows, int out_cols,
                          char* smem) {
  uint16_t* As = reinterpret_cast<uint16_t*>(smem);
  uint16_t* Bs = As + 2 * BM * BK;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;

  constexpr int AV = BM * BK / 8 / NTH;  // 16-byte vectors per thread (A)
  constexpr int BV = BN * BK / 8 / NTH;  // (B)
  u32x4_t ra[AV], rb[BV];

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      int v = tid + i * NTH, row = v >> 3, c = v & 7;
      u32x4_t z = {0u, 0u, 0u, 0u};
      ra[i] = row < a_rows ? *reinterpret_cast<const u32x4_t*>(A + (size_t)row * lda + k0 + c * 8) : z;
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      int v = tid + i * NTH, row = v >> 3, c = v & 7;
      u32x4_t z = {0u, 0u, 0u, 0u};
      rb[i] = row < b_rows ? *reinterpret_cast<const u32x4_t*>(B + (size_t)row * ldb + k0 + c * 8) : z;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      int v = tid + i * NTH, row = v >> 3, c = v & 7;
      *reinterpret_cast<u32x4_t*>(As + buf * BM * BK + swz(row, c)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      int v = tid + i * NTH, row = v >> 3, c = v & 7;
      *reinterpret_cast<u32x4_t*>(Bs + buf * BN * BK + swz(row, c)) = rb[i];
    }
  };

  f32x16_t acc[2][4];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;

  const int nk = Kd / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int ks = 0; ks < nk; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < nk) gload((ks + 1) * BK);
    const uint16_t* as = As + buf * BM * BK;
    const uint16_t* bs = Bs + buf * BN * BK;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int c = kk * 2 + (lane >> 5);
      bf16x8_t af[2], bfr[4];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        int row = wm * 64 + mb * 32 + (lane & 31);
        af[mb] = *reinterpret_cast<const bf16x8_t*>(as + swz(row, c));
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        int row = wn * 128 + nb * 32 + (lane & 31);
        bfr[nb] = *reinterpret_cast<const bf16x8_t*>(bs + swz(row, c));
      }
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb], acc[mb][nb], 0, 0, 0);
    }
    if (ks + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // epilogue: stage the bf16 tile in LDS, then write 16-byte rows
  constexpr int OC = EPI == 0 ? BN / 2 : BN;
  constexpr int CST = OC + 8;
  uint16_t* Cs = reinterpret_cast<uint16_t*>(smem);
  const int j = lane & 31;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = wm * 64 + mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (EPI == 0) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          float g = acc[mb][2 * p][r];
          float u = acc[mb][2 * p + 1][r];
          float hv = (g / (1.0f + __expf(-g))) * u;
          Cs[row * CST + wn * 64 + p * 32 + j] = (uint16_t)f32_to_bf16(hv);
        }
      } else {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          Cs[row * CST + wn * 128 + nb * 32 + j] = (uint16_t)f32_to_bf16(acc[mb][nb][r]);
      }
    }
  __syncthreads();
  constexpr int VPR = OC / 8;
  for (int v = tid; v < BM * VPR; v += NTH) {
    int row = v / VPR, col = (v % VPR) * 8;
    if (row < out_rows && col < out_cols)
      *reinterpret_cast<u32x4_t*>(out + (size_t)row * ldo + col) =
          *reinterpret_cast<const u32x4_t*>(Cs + row * CST + col);
  }
  __syncthreads();
}

// ===========================================================================
// Schedule of one launch for chunk count K (built by every workgroup in LDS).
// Segment seg < E_l is local expert seg; seg >= E_l is shared expert seg-E_l.
// ===========================================================================
struct Sched {
  int K, nseg, G;        // chunks, segments, groups = K*2*nseg
  int n_comp, n_disp, n_comb;
  int c, n_steal, final_all;
  int bnd[MAX_K + 1];    // chunk token boundaries ceil(q*T/K)
  int cstart[MAX_K + 1]; // combine units before chunk q
  int g1need[MAX_K];     // GEMM1 tiles of chunk q
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
  int part[NTH];
  int sl[DT * MAX_TOPK];
  float wt[CT * MAX_TOPK];
};

// block-wide exclusive scan of n ints in LDS (all threads call): each thread
// sums a contiguous run, wavefront shuffles scan the run sums, then the runs
// are rewritten with their offsets
__device__ void block_exscan(int* v, int n, int* part) {
  const int tid = threadIdx.x;
  const int lane = tid & (WAVE - 1), wave = tid / WAVE;
  const int per = (n + NTH - 1) / NTH;
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

__device__ void build_sched(const FwdArgs& a, Sched& S, Scratch& W, int K) {
  const int tid = threadIdx.x;
  const int ki = kopt_index(K);
  const int nseg = a.El + a.S;
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
  for (int v = tid; v < K * nseg; v += NTH) {
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
  // group sizes in queue order: chunk, then phase (GEMM0, GEMM1), then segment
  for (int gi = tid; gi < S.G; gi += NTH) {
    int q = gi / (2 * nseg), ph = (gi / nseg) & 1, seg = gi % nseg;
    S.gstart[gi] = S.mb[q * nseg + seg] * (ph ? a.nt1 : a.nt0);
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
// Movement work: dispatch (x rows -> expert-contiguous A slots, each row read
// once and written to all its local slots) and combine (weighted sum of the
// expert outputs of each token into the output staging region).
// ===========================================================================
__device__ void dispatch_unit(const FwdArgs& a, const Sched* S, Scratch& W, int u, bool signal) {
  const int tid = threadIdx.x;
  const int g0 = u * DT;
  const int nt = min(DT, a.T - g0);
  const int k = a.k;
  for (int i = tid; i < nt * k; i += NTH) W.sl[i] = a.slot[(size_t)g0 * k + i];
  __syncthreads();
  const int VPR = a.H >> 3;
  const int total = nt * VPR;
  for (int v0 = tid; v0 < total; v0 += 4 * NTH) {
    u32x4_t val[4];
    int tt[4], cc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int v = v0 + i * NTH;
      tt[i] = -1;
      if (v < total) {
        int t = v / VPR;
        int c = v - t * VPR;
        bool any = false;
        for (int j = 0; j < k; ++j) any |= (unsigned)W.sl[t * k + j] < (unsigned)a.xmax;
        if (any) {
          tt[i] = t;
          cc[i] = c;
          val[i] = *reinterpret_cast<const u32x4_t*>(a.x + (size_t)(g0 + t) * a.H + c * 8);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (tt[i] < 0) continue;
      for (int j = 0; j < k; ++j) {
        int s = W.sl[tt[i] * k + j];
        if ((unsigned)s < (unsigned)a.xmax) *reinterpret_cast<u32x4_t*>(a.A + (size_t)s * a.H + cc[i] * 8) = val[i];
      }
    }
  }
  if (signal) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid < WAVE) {
      fence_release_agent();
      for (int i = tid; i < nt * k; i += WAVE) {
        int s = W.sl[i];
        if ((unsigned)s >= (unsigned)a.xmax) continue;
        int g = g0 + i / k;
        int le = a.topk_idx[(size_t)g * k + (i % k)] - a.e0;
        if ((unsigned)le >= (unsigned)a.El) continue;
        int q = (int)(((long long)g * S->K) / a.T);
        int id = S->mb[q * S->nseg + le] + (s - S->row0[q * S->nseg + le]) / BM;
        if ((unsigned)id < (unsigned)a.mt_max) fetch_add_relaxed(&a.ctl[CTL_READY + id], 1);
      }
    }
  }
  __syncthreads();
}

__device__ void combine_tokens(const FwdArgs& a, Scratch& W, int g0, int nt) {
  const int tid = threadIdx.x;
  const int k = a.k;
  for (int i = tid; i < nt * k; i += NTH) {
    W.sl[i] = a.slot[(size_t)g0 * k + i];
    W.wt[i] = a.topk_w[(size_t)g0 * k + i];
  }
  __syncthreads();
  const int VPR = a.H >> 3;
  const int total = nt * VPR;
  for (int v = tid; v < total; v += NTH) {
    int t = v / VPR, c = v - t * VPR;
    int g = g0 + t;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
    for (int j = 0; j < k; ++j) {
      int s = W.sl[t * k + j];
      if ((unsigned)s >= (unsigned)a.xmax) continue;
      float w = W.wt[t * k + j];
      u32x4_t o = *reinterpret_cast<const u32x4_t*>(a.O + (size_t)s * a.H + c * 8);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += w * bf16_lo(o[q]);
        acc[2 * q + 1] += w * bf16_hi(o[q]);
      }
    }
    if (g < a.Tr) {
      for (int s = 0; s < a.S; ++s) {
        u32x4_t o = *reinterpret_cast<const u32x4_t*>(a.O + (size_t)(a.xmax + s * a.Tr + g) * a.H + c * 8);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] += bf16_lo(o[q]);
          acc[2 * q + 1] += bf16_hi(o[q]);
        }
      }
    }
    u32x4_t r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = pack_bf16x2(acc[2 * q], acc[2 * q + 1]);
    *reinterpret_cast<u32x4_t*>(a.y + (size_t)g * a.H + c * 8) = r;
  }
  __syncthreads();
}

// ===========================================================================
// Compute work: one tile of GEMM0 (+SiLU*up) or GEMM1 for (chunk, segment,
// row tile, column tile).  Within a group the row tile runs fastest, so
// consecutive claims share the same weight columns.
// ===========================================================================
struct TileRef {
  int q, ph, seg, mt, nt, rows;
};

__device__ __forceinline__ TileRef decode_tile(const FwdArgs& a, const Sched& S, int t) {
  int lo = 0, hi = S.G;  // find last gi with gstart[gi] <= t
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
  r.mt = local % nmt;
  r.nt = local / nmt;
  r.rows = min(BM, rows - r.mt * BM);
  return r;
}

__device__ void run_gemm(const FwdArgs& a, const Sched& S, const TileRef& r, char* smem) {
  const int qs = r.q * S.nseg + r.seg;
  const size_t orow = (size_t)S.row0[qs] + (size_t)r.mt * BM;
  const int n0 = r.nt * BN;
  if (r.ph == 0) {
    const size_t arow = (size_t)S.arow0[qs] + (size_t)r.mt * BM;
    const uint16_t* Aop = (r.seg < a.El ? a.A : a.x) + arow * a.H;
    const size_t two_f = 2 * (size_t)a.F;
    const uint16_t* Bop = a.w13 + (size_t)r.seg * two_f * a.H + (size_t)n0 * a.H;
    uint16_t* out = a.Hb + orow * a.F + n0 / 2;
    gemm_tile<0>(Aop, a.H, r.rows, Bop, a.H, (int)(two_f - n0), a.H, out, a.F, r.rows, a.F - n0 / 2,
                 smem);
  } else {
    const uint16_t* Aop = a.Hb + orow * a.F;
    const uint16_t* Bop = a.w2t + (size_t)r.seg * a.H * a.F + (size_t)n0 * a.F;
    uint16_t* out = a.O + orow * a.H + n0;
    gemm_tile<1>(Aop, a.F, r.rows, Bop, a.F, a.H - n0, a.F, out, a.H, r.rows, a.H - n0, smem);
  }
}

// ===========================================================================
// Prologue: the routing-derived workload and the plan (sections 3.1-3.3),
// computed redundantly by every workgroup from a small read of the stats.
// ===========================================================================
__device__ void prologue_plan(const FwdArgs& a, Sched& S, Scratch& W) {
  const int tid = threadIdx.x;
  const int nseg = a.El + a.S;
  if (tid < KOPT) W.ntk[tid] = 0;
  __syncthreads();
  // GEMM tiles at each stored chunk option (for W_tile of Eq 14)
  for (int ki = 0; ki < KOPT; ++ki) {
    const int K = kopt_value(ki);
    long long part = 0;
    for (int v = tid; v < K * nseg; v += NTH) {
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
      part += (long long)ceil_div(rows, BM) * (a.nt0 + a.nt1);
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

__device__ bool wait_geq(const FwdArgs& a, Scratch& W, const int* p, int target) {
  if (a.inject_stall) target += 1 << 30;
  if (threadIdx.x == 0) {
    int ok = 1;
    if (ld_acquire(p) < target) {
      const uint64_t deadline = now_ticks() + (uint64_t)a.timeout_ticks;
      while (ld_acquire(p) < target) {
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

__device__ __forceinline__ void signal_done(int* p) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(p, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// returns false when the launch was aborted
__device__ bool run_compute_tile(const FwdArgs& a, const Sched& S, Scratch& W, int t, char* smem) {
  TileRef r = decode_tile(a, S, t);
  const int id = S.mb[r.q * S.nseg + r.seg] + r.mt;
  if (r.ph == 0) {
    if (r.seg < a.El && !wait_geq(a, W, &a.ctl[CTL_READY + id], r.rows)) return false;
    run_gemm(a, S, r, smem);
    signal_done(&a.ctl[CTL_READY + a.mt_max + id]);
  } else {
    if (!wait_geq(a, W, &a.ctl[CTL_READY + a.mt_max + id], a.nt0)) return false;
    run_gemm(a, S, r, smem);
    signal_done(&a.ctl[CTL_G1DONE + r.q]);
  }
  return true;
}

__device__ bool combine_loop(const FwdArgs& a, const Sched& S, Scratch& W) {
  for (;;) {
    int u = claim(W, &a.ctl[CTL_Q_COMB]);
    if (u >= S.n_comb) return true;
    int q = 0;
    while (q + 1 < S.K && S.cstart[q + 1] <= u) ++q;
    if (!wait_geq(a, W, &a.ctl[CTL_G1DONE + q], S.g1need[q])) return false;
    int g0 = S.bnd[q] + (u - S.cstart[q]) * CT;
    int nt = min(CT, S.bnd[q + 1] - g0);
    combine_tokens(a, W, g0, nt);
  }
}

// ===========================================================================
// The persistent megakernel: one workgroup per CU, co-resident (cooperative
// launch).  The first c workgroups to arrive become movement workers.
// ===========================================================================
__global__ void __launch_bounds__(NTH, 1) moe_megakernel(FwdArgs a) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(16))) char smem[GEMM_SMEM];
  const int tid = threadIdx.x;

  if (blockIdx.x == 0)
    for (int i = tid; i < a.ctl_words; i += NTH) a.ctl_next[i] = 0;

  prologue_plan(a, S, W);
  build_sched(a, S, W, S.K);

  if (tid == 0) W.bc[0] = fetch_add_relaxed(&a.ctl[CTL_TICKET], 1);
  __syncthreads();
  const bool mover = W.bc[0] < S.c;
  __syncthreads();

  if (mover) {
    // dispatch: every token row, in token (hence chunk) order
    for (;;) {
      int u = claim(W, &a.ctl[CTL_Q_DISP]);
      if (u >= S.n_disp) break;
      dispatch_unit(a, &S, W, u, true);
    }
    // bubble stealing: n_steal GEMM tiles right after dispatch (section 3.2.2)
    for (int i = 0; i < S.n_steal; ++i) {
      int t = claim(W, &a.ctl[CTL_Q_COMP]);
      if (t >= S.n_comp) break;
      if (!run_compute_tile(a, S, W, t, smem)) return;
    }
    combine_loop(a, S, W);
  } else {
    for (;;) {
      int t = claim(W, &a.ctl[CTL_Q_COMP]);
      if (t >= S.n_comp) break;
      if (!run_compute_tile(a, S, W, t, smem)) return;
    }
    // final combine on every worker (section 4)
    if (S.final_all) combine_loop(a, S, W);
  }
}

// ===========================================================================
// Serial baseline: four kernels, each on every CU, no overlap.
// ===========================================================================
__global__ void __launch_bounds__(NTH, 1) serial_dispatch_kernel(FwdArgs a) {
  __shared__ Scratch W;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0)
    for (int i = tid; i < a.ctl_words; i += NTH) a.ctl_next[i] = 0;
  const int n = ceil_div(a.T, DT);
  for (;;) {
    int u = claim(W, &a.ctl[CTL_SQ + 0]);
    if (u >= n) break;
    dispatch_unit(a, nullptr, W, u, false);
  }
}

template <int PH>
__device__ void serial_gemm(const FwdArgs& a, int qslot) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(16))) char smem[GEMM_SMEM];
  build_sched(a, S, W, 1);
  const int first = S.gstart[PH * S.nseg];
  const int count = S.gstart[(PH + 1) * S.nseg] - first;
  for (;;) {
    int t = claim(W, &a.ctl[CTL_SQ + 64 * qslot]);
    if (t >= count) break;
    TileRef r = decode_tile(a, S, first + t);
    run_gemm(a, S, r, smem);
  }
}

__global__ void __launch_bounds__(NTH, 1) serial_gemm0_kernel(FwdArgs a) { serial_gemm<0>(a, 1); }
__global__ void __launch_bounds__(NTH, 1) serial_gemm1_kernel(FwdArgs a) { serial_gemm<1>(a, 2); }

__global__ void __launch_bounds__(NTH, 1) serial_combine_kernel(FwdArgs a) {
  __shared__ Scratch W;
  const int n = ceil_div(a.T, CT);
  for (;;) {
    int u = claim(W, &a.ctl[CTL_SQ + 192]);
    if (u >= n) break;
    int g0 = u * CT;
    combine_tokens(a, W, g0, min(CT, a.T - g0));
  }
}

}  // namespace moe
