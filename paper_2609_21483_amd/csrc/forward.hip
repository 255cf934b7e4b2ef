// The MoE layer on one GPU's share (paper section 2.1, Fig 3), run either as
// one persistent megakernel with movement and compute workers (sections 3-4)
// or as four separate kernels (the serial baseline, "w/o S+T" of section 5.6).
//
// Data layout in HBM
//   x    bf16 [T][H]        staging regions: rank r's rows at r*Tr
//   A    bf16 [rows][H]     dispatched rows, expert-contiguous, then chunk-
//                           contiguous within an expert (slot order within a
//                           chunk); every (expert, chunk) starts on a 32-row
//                           group (row_off); group-tiled (gemm::AOp)
//   Hbuf bf16 [rows][F]     SiLU(gate)*up per row (shared experts after the
//                           routed rows), the same row map, group-tiled
//   O    bf16 [rows][H]     expert outputs per row, the same row map
//   part fp32 [split][X+S*Tr+pad][H]  split-K partials of GEMM1 (when split)
//   y    bf16 [T][H]        output staging regions
//   w13  bf16 [E_l+S][2F][H] gate/up weights, k-contiguous, 32-col interleave,
//                           slab-tiled (common.h)
//   w2t  bf16 [E_l+S][H][F]  down weights, k-contiguous, slab-tiled
#include <type_traits>

#include "common.h"
#include "gemm.h"
#include "kernels.h"

namespace moe {

constexpr int NWF = FNTH / WAVE;  // waves per forward workgroup

// ===========================================================================
// Schedule of one launch for chunk count K (struct Sched, kernels.h): built
// once per K option by sched_build_kernel when the routing tables are, and
// copied into each workgroup's LDS by its prologue.
// ===========================================================================


struct Scratch {
  int bc[8];
  DevCalib cal;                                        // the calibration table, staged by the prologue
  int st[ST_WORDS];                                    // routing stats (ST_*), staged by the prologue
  int part[NWF];
  int wsl[NWF][WAVE];    // per wavefront: slots of its unit's (token, j) pairs
  int wact[NWF][DT];     // per wavefront: its dispatch unit's tokens that have a local slot
  int dexh;              // every dispatch unit has been claimed (seen by this workgroup)
  int ticket;            // this workgroup's arrival ticket (trace records)
  int tcnt[NWF];         // trace records written by each wavefront
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

// XCD-aware tile queues.  A tile's weight slab is its GEMM0 column tile, or
// its GEMM1 (column tile, split) pair; the tiles of one slab share the slab's
// weights, so they are queued for one XCD (slab class = slab mod NXCD) and
// read them from that XCD's L2.  Stage = (chunk, phase) in DAG order; each
// stage has one queue per class, the row tile fastest within a slab.
__device__ __forceinline__ int phase_slabs(const FwdArgs& a, int ph) { return ph == 0 ? a.nt0 : a.nt1 * a.nsplit; }
__device__ __forceinline__ int class_slabs(int ns, int x) { return ns > x ? (ns - x + NXCD - 1) / NXCD : 0; }

// Readiness levels order the row tiles of a stage by when their inputs can be
// complete.  Dispatch writes a local expert's rows in token order, so row
// tile mt of a segment of `rows` rows is complete once the fraction
// min((mt + 1) * BM, rows) / rows of the segment is written; its level is
// that fraction rounded up to a multiple of 1/NLVL (1..NLVL).  Shared-expert
// rows are read straight from x: level 0, ready at launch.  With every
// worker copying rows at the start, the routed row tiles all complete at
// nearly the same time, and one routed level (NLVL = 1) measures fastest:
// it keeps the row tiles of one expert and weight slab together, so the
// tiles running on an XCD share that slab in its L2 (finer levels spread the
// first claims over every expert and slab and fetch the weights several
// times over).
__device__ __forceinline__ int tiles_upto(int rows, int L) {  // routed tiles at level <= L
  const int nmt = (rows + BM - 1) / BM;
  if (L <= 0) return 0;
  if (L >= NLVL) return nmt;
  return min(nmt, (int)(((long long)L * rows) / ((long long)NLVL * BM)));
}
__device__ __forceinline__ int level_lo(int rows, bool shared, int L) {  // first row tile of level L
  return shared ? 0 : tiles_upto(rows, L - 1);
}
__device__ __forceinline__ int level_tiles(int rows, bool shared, int L) {
  if (shared) return L == 0 ? (rows + BM - 1) / BM : 0;
  return tiles_upto(rows, L) - tiles_upto(rows, L - 1);
}

// Queue order of the stages (chunk, phase) of a K-chunk schedule, skewed by
// one chunk: (0,G0), (1,G0), (0,G1), (2,G0), (1,G1), ..., (K-1,G0), (K-2,G1),
// (K-1,G1).  Workers reach chunk q's GEMM1 tiles only after claiming chunk
// q+1's GEMM0 tiles, which depend on dispatch alone, so chunk q's last GEMM0
// tiles finish while those run instead of holding up a worker at every chunk
// boundary.  Returns chunk << 1 | phase.
__device__ __forceinline__ int stage_qph(int s, int K) {
  if (s == 0) return 0;
  if (s >= 2 * K - 1) return ((K - 1) << 1) | 1;
  const int j = (s + 1) >> 1;
  return (s & 1) ? (j << 1) : (((j - 1) << 1) | 1);
}

// The schedule for K in S (all threads call; sched_build_kernel's workgroups).
// sub, rof: the chunk sub-offset and row-map tables (a.sub_off, a.row_off)
__device__ __forceinline__ void build_sched(const FwdArgs& a, const int* sub, const int* rof, Sched& S, Scratch& W,
                                            int K) {
  const int tid = threadIdx.x;
  const int ki = kopt_index(K);
  const int nseg = a.El + a.S;
  const int g1tiles = a.nt1 * a.nsplit;  // GEMM1 tiles per row tile
  // chunk token boundaries ceil(q T / K); K is 1, 2, 4 or 8
  if (tid <= K) S.bnd[tid] = (int)(((long long)tid * a.T + K - 1) >> __builtin_ctz((unsigned)K));
  if (tid == 0) {
    S.K = K;
    S.nseg = nseg;
    S.G = K * 2 * nseg;
    S.n_comb = ceil_div(a.T, a.ct);
    S.n_disp = ceil_div(a.T, a.dt);
  }
  __syncthreads();
  for (int v = tid; v < K * nseg; v += FNTH) {
    int q = v / nseg, seg = v % nseg;
    int rows, sbase, arow0;
    const int row0 = rof[((size_t)ki * nseg + seg) * SUBW + q];
    if (seg < a.El) {
      const int* so = sub + ((size_t)ki * a.El + seg) * SUBW;
      sbase = so[q];
      rows = so[q + 1] - so[q];
      arow0 = row0;
    } else {
      int t0 = S.bnd[q], t1 = min(S.bnd[q + 1], a.Tr);
      rows = max(0, t1 - t0);
      sbase = t0;
      arow0 = t0;
    }
    S.rows[v] = rows;
    S.row0[v] = row0;
    S.sbase[v] = sbase;
    S.arow0[v] = arow0;
    S.mb[v] = ceil_div(rows, BM);
  }
  __syncthreads();
  for (int gi = tid; gi < S.G; gi += FNTH) {
    int q = gi / (2 * nseg), ph = (gi / nseg) & 1, seg = gi % nseg;
    S.gstart[gi] = S.mb[q * nseg + seg] * (ph ? g1tiles : a.nt0);
  }
  if (tid == 0) S.gstart[S.G] = 0;
  __syncthreads();
  for (int v = tid; v < 2 * K * NXCD; v += FNTH) {
    const int stage = v / NXCD, x = v % NXCD, qp = stage_qph(stage, K), q = qp >> 1;
    const int nsx = class_slabs(phase_slabs(a, qp & 1), x);
    int n = 0;
    for (int seg = 0; seg < nseg; ++seg) n += nsx * ceil_div(S.rows[q * nseg + seg], BM);
    S.ncls[stage][x] = n;
  }
  for (int v = tid; v < K * (NLVL + 1); v += FNTH) {
    const int q = v / (NLVL + 1), L = v % (NLVL + 1);
    int n = 0;
    for (int seg = 0; seg < nseg; ++seg) n += level_tiles(S.rows[q * nseg + seg], seg >= a.El, L);
    S.lvl[q][L] = n;
  }
  __syncthreads();
  if (tid < K)
    for (int L = 1; L <= NLVL; ++L) S.lvl[tid][L] += S.lvl[tid][L - 1];
  block_exscan(S.mb, K * nseg, W.part);
  block_exscan(S.gstart, S.G + 1, W.part);
  if (tid == 0) S.n_comp = S.gstart[S.G];
  __syncthreads();
}

// A launch's schedule for chunk count K: the stored image (built by
// sched_build_kernel when the routing tables were) copied into S after the
// plan fields, which it leaves alone.  All threads call; ends with a barrier.
__device__ __forceinline__ void load_sched(const FwdArgs& a, Sched& S, int K) {
  const int32_t* src = a.sched + (size_t)kopt_index(K) * SCHED_WORDS;
  int* dst = reinterpret_cast<int*>(&S);
  constexpr int N4 = (SCHED_WORDS - SCHED_IMG0) / 4;
  static_assert(SCHED_IMG0 % 4 == 0 && SCHED_WORDS % 4 == 0, "16-byte copies");
  for (int i = threadIdx.x; i < N4; i += FNTH)
    reinterpret_cast<u32x4_t*>(dst + SCHED_IMG0)[i] = reinterpret_cast<const u32x4_t*>(src + SCHED_IMG0)[i];
  __syncthreads();
}

// ===========================================================================
// Movement work, one wavefront per unit (no workgroup barriers, so the eight
// wavefronts of a movement worker overlap their latency chains):
// dispatch copies the rows of dt tokens into their expert-contiguous A slots
// (each row read once, written to every local slot); combine writes the
// weighted sum of the expert outputs of ct tokens into the output staging
// region.
// ===========================================================================
__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE); }

// ---- timeline trace (off when a.trace is NULL) ------------------------------
__device__ __forceinline__ int xcd_id() {
  int v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(v));
  return v;
}

// Test hook (moe_set_jitter): a pseudo-random delay of 0..jitter_max sleeps
// of 64 cycles, drawn from (seed, workgroup, wavefront, event), so that
// workgroups reach their claims in perturbed orders.
__device__ __forceinline__ void jitter(const FwdArgs& a, uint32_t event) {
  if (!a.jitter_max) return;
  uint32_t h = a.jitter_seed ^ (blockIdx.x * 0x9E3779B1u) ^ (event * 0x85EBCA77u) ^
               ((uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * 0xC2B2AE3Du);
  h ^= h >> 16;
  h *= 0x7FEB352Du;
  h ^= h >> 15;
  h *= 0x846CA68Bu;
  h ^= h >> 16;
  const int n = __builtin_amdgcn_readfirstlane((int)(h % (uint32_t)(a.jitter_max + 1)));
  for (int i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(1);
}

// One lane of a wavefront appends one record to the wavefront's own segment
// of the trace buffer (segment blockIdx.x * NWF + wave, trace_cap records):
// a per-wavefront LDS counter, no global atomics, so tracing does not
// serialise the workgroups on a shared counter.
__device__ __forceinline__ void trace_rec(const FwdArgs& a, Scratch& W, int kind, int ticket, long long id,
                                          uint64_t t0, uint64_t t1, uint64_t t2) {
  if (!a.trace) return;
  const int wv = wave_id();
  const int slot = W.tcnt[wv]++;
  if (slot >= a.trace_cap) return;
  long long* r = a.trace + a.trace_rec0 + ((size_t)(blockIdx.x * NWF + wv) * a.trace_cap + slot) * 4;
  r[0] = (long long)kind | ((long long)ticket << 8) | ((long long)xcd_id() << 20) | (id << 32);
  r[1] = (long long)t0;
  r[2] = (long long)t1;
  r[3] = (long long)t2;
}

// Dispatch units in the megakernel: the first round is owned statically,
// wavefront w of the worker with ticket t copying unit t * NWF + w (every
// worker that moves rows at launch: all of them when compute workers steal
// movement, else the movement workers), so the launch starts without queue
// traffic; units are sized so that this round covers all of them whenever T
// allows.  Later units are claimed from the sharded queue (claim_unit).

// Dispatch (section 4, with dedup): a wavefront copies the rows of tokens
// [u*dt, u*dt + dt) of unit u; each token row is read once and written to
// every local slot it has.  Only tokens with a local slot are read.
// In the megakernel (SIG) the rows are written with agent-coherent (sc1)
// 16-byte buffer stores, so once they have completed (vmcnt 0) they are
// visible to every XCD and the readiness counters can be raised without an
// L2 write-back; the serial kernel, which ends at a kernel boundary, uses
// plain stores.  Either way the wavefront drains its stores before its next
// unit, which measures faster on this GPU than letting them queue.

// Row in A / Hbuf / O of the local pair (g, j) with slot s >= 0 of local
// expert le: its (expert, chunk) segment's first row plus its place in the
// segment (common.h).  With the launch's schedule S the segment comes from
// LDS; without one (the separate kernels) from the tables, for serial_K.
__device__ __forceinline__ int pair_row(const FwdArgs& a, const Sched* S, int g, int le, int s) {
  if (S) {
    const int v = (int)(((long long)g * S->K) / a.T) * S->nseg + le;
    return S->row0[v] + (s - S->sbase[v]);
  }
  const int K = a.serial_K, ki = kopt_index(K), q = (int)(((long long)g * K) / a.T);
  return a.row_off[(ki * (a.El + a.S) + le) * SUBW + q] + (s - a.sub_off[(ki * a.El + le) * SUBW + q]);
}

// Row in Hbuf / O of token g (g < Tr) of shared expert sh.
__device__ __forceinline__ int shared_row(const FwdArgs& a, const Sched* S, int g, int sh) {
  if (S) {
    const int q = (int)(((long long)g * S->K) / a.T), v = q * S->nseg + a.El + sh;
    return S->row0[v] + (g - S->sbase[v]);
  }
  const int K = a.serial_K, ki = kopt_index(K), q = (int)(((long long)g * K) / a.T);
  const int t0 = (int)(((long long)q * a.T + K - 1) / K);
  return a.row_off[(ki * (a.El + a.S) + a.El + sh) * SUBW + q] + (g - t0);
}

// this lane's A row of unit u (lane = token * k + j), or -1 when the pair is
// not local
__device__ __forceinline__ int unit_row(const FwdArgs& a, const Sched* S, int u) {
  const int g0 = u * a.dt;
  const int lane = lane_id();
  if (g0 >= a.T || lane >= min(a.dt, a.T - g0) * a.k) return -1;
  const int g = g0 + lane / a.k;
  const int s = a.slot[(size_t)g0 * a.k + lane];
  return s < 0 ? -1 : pair_row(a, S, g, a.topk_idx[(size_t)g0 * a.k + lane] - a.e0, s);
}

// The lane id and the launch constants of a movement unit are defined by
// opaque statements (see gemm::opaque), so that where a unit runs inside the
// GEMM tile loop (movement stealing) the optimiser cannot hoist the unit's
// per-lane index and address arithmetic out of that loop and keep it live
// across the GEMM mainloop.
using gemm::lane_here;

template <bool SIG>
__device__ __forceinline__ void dispatch_copy(const FwdArgs& a, Scratch& W, int u, int cur) {
  using gemm::opaque;
  constexpr int VB = 32;  // 16-byte vectors per lane in flight
  const int lane = lane_here();
  const int wv = opaque(wave_id());
  int* sl = W.wsl[wv];
  int* act = W.wact[wv];
  const int k = opaque(a.k);
  const int H = opaque(a.H);
  const int VPR = H >> 3;
  const int T = opaque(a.T);
  const int dt = opaque(a.dt);
  const int g0 = u * dt;
  const int nt = min(dt, T - g0);
  sl[lane] = cur;
  // tokens with at least one local slot, compacted in token order
  const uint64_t vm = __builtin_amdgcn_ballot_w64(cur >= 0);
  const bool tact = lane < nt && ((vm >> min(lane * k, 56)) & ((1ull << k) - 1)) != 0;
  const uint64_t am = __builtin_amdgcn_ballot_w64(tact);
  const int na = __builtin_popcountll(am);
  if (tact) act[__builtin_amdgcn_mbcnt_hi((uint32_t)(am >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)am, 0))] = lane;
  __builtin_amdgcn_wave_barrier();
  // A spans less than 4 GiB (checked on the host), so 32-bit byte offsets
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(a.A, 0, -1, 0x00020000);
  const int total = na * VPR;
  for (int v0 = lane; v0 < total; v0 += VB * WAVE) {
    u32x4_t val[VB];
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = v0 + i * WAVE;
      if (v < total) {
        int t = 0;
#pragma unroll
        for (int m = 1; m < DT; ++m) t += v >= m * VPR;
        const int c = v - t * VPR;
        val[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.x + (size_t)(g0 + act[t]) * H) + c);
      }
    }
    // every load of the pass has landed: the stores below (a run-time number
    // per vector) then issue back to back.  Without this drain the compiler
    // cannot count the stores in flight between a load and its use, and
    // waits for all of them (vmcnt counts stores too) before every vector.
    gemm::wait_vm<0>();
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = v0 + i * WAVE;
      if (v >= total) continue;
      int t = 0;
#pragma unroll
      for (int m = 1; m < DT; ++m) t += v >= m * VPR;
      const int c = v - t * VPR;
      const int tok = act[t];
      for (int j = 0; j < k; ++j) {
        const int s = sl[tok * k + j];
        if (s < 0) continue;
        // A is group-tiled (gemm::AOp): 16-byte chunk c of row s lies in
        // k-step block c / 4 of group s / 32, at row s % 32 of the block
        const uint32_t off = ((uint32_t)(s >> 5) * (uint32_t)H * 32u + (uint32_t)(c >> 2) * 1024u +
                              (uint32_t)(s & 31) * 32u + (uint32_t)(c & 3) * 8u) * 2u;
        if constexpr (SIG) {
          __builtin_amdgcn_raw_buffer_store_b128(val[i], rA, off, 0, 16 /* sc1 */);
        } else {
          *reinterpret_cast<u32x4_t*>(reinterpret_cast<char*>(a.A) + off) = val[i];
        }
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
}

// Readiness accounting of a copied unit whose rows have reached the coherence
// point (needs the schedule): each row tile the unit wrote rows of gains
// that many rows, one counter update per distinct row tile.
__device__ __forceinline__ void dispatch_count(const FwdArgs& a, const Sched* S, int u, int cur) {
  using gemm::opaque;
  const int lane = lane_here();
  const int k = opaque(a.k);
  const int T = opaque(a.T);
  const int g0 = u * opaque(a.dt);
  int id = -1;
  if (cur >= 0) {
    const int g = g0 + lane / k;
    const int le = a.topk_idx[(size_t)g * k + (lane % k)] - a.e0;
    if ((unsigned)le < (unsigned)a.El) {
      const int q = (int)(((long long)g * S->K) / T);
      id = S->mb[q * S->nseg + le] + (cur - S->row0[q * S->nseg + le]) / BM;
      if ((unsigned)id >= (unsigned)a.mt_max) id = -1;
    }
  }
  uint64_t pending = __builtin_amdgcn_ballot_w64(id >= 0);
  while (pending) {
    const int leader = __builtin_ctzll(pending);
    const int tile = __builtin_amdgcn_readlane(id, leader);
    const uint64_t same = __builtin_amdgcn_ballot_w64(id == tile);
    if (lane == leader) fetch_add_relaxed(&a.ctl[CTL_READY + tile * CTL_PAD], (int)__builtin_popcountll(same));
    pending &= ~same;
  }
}

// A whole unit: copy, then (megakernel) count.
template <bool SIG>
__device__ __forceinline__ void dispatch_one(const FwdArgs& a, const Sched* S, Scratch& W, int u, int cur) {
  const uint64_t tr0 = (SIG && a.trace) ? now_ticks() : 0;
  dispatch_copy<SIG>(a, W, u, cur);
  if constexpr (SIG) {
    const uint64_t tr1 = a.trace ? now_ticks() : 0;
    dispatch_count(a, S, u, cur);
    if (a.trace && lane_id() == 0) trace_rec(a, W, 5, W.ticket, u | ((long long)wave_id() << 24), tr0, tr1, now_ticks());
  }
  __builtin_amdgcn_wave_barrier();
}

// serial kernel: units u0, u0 + ustride, ..., the next unit's slot entries
// fetched while the current one is copied
__device__ __forceinline__ void dispatch_static(const FwdArgs& a, Scratch& W, int u, int ustride) {
  const int nu = ceil_div(a.T, a.dt);
  int next = unit_row(a, nullptr, u);
  for (; u < nu; u += ustride) {
    const int cur = next;
    next = unit_row(a, nullptr, u + ustride);
    dispatch_one<false>(a, nullptr, W, u, cur);
  }
}

// Megakernel: movement units are claimed per wavefront from NSHARD queues
// at ctl[base + shard * CTL_PAD] (unit u is the (u / NSHARD)-th of shard
// u % NSHARD, so every shard advances in token order).  Lane l reads the
// head of shard (shard + l) % NSHARD, all in one vector read; the nearest
// shard with units left takes one atomic.  A shard found exhausted by that
// atomic reads exhausted from then on, so the loop ends within NSHARD
// rounds.  Returns the unit, or -1 once every shard is exhausted.
static_assert(NSHARD == WAVE, "one queue shard per lane");
__device__ __forceinline__ int claim_unit(const FwdArgs& a, int base, int n_units, int& shard) {
  const int lane = lane_id();
  for (int round = 0; round < NSHARD; ++round) {
    const int sl = (shard + lane) & (NSHARD - 1);
    const bool open = ld_relaxed(&a.ctl[base + sl * CTL_PAD]) * NSHARD + sl < n_units;
    const uint64_t m = __builtin_amdgcn_ballot_w64(open);
    if (!m) return -1;
    shard = (shard + (int)__builtin_ctzll(m)) & (NSHARD - 1);
    int v = 0;
    if (lane == 0) v = fetch_add_relaxed(&a.ctl[base + shard * CTL_PAD], 1);
    const int u = __builtin_amdgcn_readfirstlane(v) * NSHARD + shard;
    if (u < n_units) return u;
  }
  return -1;
}

// a wavefront's first shard: spread over the shards by worker and wavefront
__device__ __forceinline__ int first_shard(const Scratch& W) { return (W.ticket * NWF + wave_id()) & (NSHARD - 1); }

// the next dispatch unit past the statically owned ones, or -1 (at once when
// every unit is owned statically: no queue reads)
__device__ __forceinline__ int claim_disp(const FwdArgs& a, const Sched& S, int& shard) {
  if (S.disp0 >= S.n_disp) return -1;
  const int v = claim_unit(a, CTL_QD, S.n_disp - S.disp0, shard);
  return v < 0 ? -1 : S.disp0 + v;
}

// movement worker: dispatch until every unit is claimed
__device__ __forceinline__ void dispatch_claimed(const FwdArgs& a, const Sched& S, Scratch& W) {
  int shard = first_shard(W);
  for (;;) {
    const int u = claim_disp(a, S, shard);
    if (u < 0) break;
    jitter(a, 0x20000u + (uint32_t)u);
    dispatch_one<true>(a, &S, W, u, unit_row(a, &S, u));
  }
}

__device__ __forceinline__ const StoredPlan* stored_plan(const FwdArgs& a) {
  return reinterpret_cast<const StoredPlan*>(a.sched + (size_t)KOPT * SCHED_WORDS);
}

// The chunk count a layer's prologue will pick without evaluating the cost
// model: the forced plan's, or the plan stored with its routing tables while
// the calibration is unchanged; 0 when it will evaluate the model (or runs
// no movement stealing).
__device__ __forceinline__ int planned_K(const FwdArgs& a) {
  if (!a.move_steal || a.mode == MOE_MODE_STATIC || a.static_disp) return 0;
  if (a.forced) return a.fplan.K;
  const StoredPlan* sp = stored_plan(a);
  return sp->gen == a.calib_gen ? sp->p.K : 0;
}

// A later layer of a stacked launch (an): its dispatch units, claimed from
// its queue by this layer's movement workers while this layer's GEMMs run
// (they depend on nothing of this layer), with that layer's schedule image
// read in place; its own workers claim what is left when they arrive.
__device__ __forceinline__ void dispatch_ahead(const FwdArgs& an, Scratch& W) {
  const int K = planned_K(an);
  if (K <= 0) return;
  const Sched* Sg = reinterpret_cast<const Sched*>(an.sched + (size_t)kopt_index(K) * SCHED_WORDS);
  const int n_disp = ceil_div(an.T, an.dt);
  int shard = first_shard(W);
  for (int u; (u = claim_unit(an, CTL_QD, n_disp, shard)) >= 0;) dispatch_one<true>(an, Sg, W, u, unit_row(an, Sg, u));
}

__device__ __forceinline__ bool wave_wait_all(const FwdArgs& a, const int* p, int target);

// One wavefront combines nt <= ct tokens.  Each token has KS = k + S source
// rows: its k routed slots (weight w, absent when the expert is not local)
// followed by its S shared-expert rows (weight 1, present for tokens of rank
// 0).  They are summed in that order in fp32.  A source row is O (bf16).  KS
// is a template constant so that every lane keeps about 16 row vectors in
// flight.
// Entries past a token's present rows (or past the unit) load from x with
// weight 0 (x is finite and never written during a launch), so they add +0
// and the loads of a pass are straight-line code that issues them all before
// the first wait (a load under a per-lane branch is preceded by a full
// drain).  They must not read O: a line of O loaded before its row tile is
// published would sit stale in this CU's L1 for the unit that needs it.
template <int KS>
__device__ __forceinline__ void combine_body(const FwdArgs& a, const int* sl, const float* wt, int g0, int nt) {
  constexpr int P = KS >= 2 ? 16 / KS : 8;  // positions per lane per pass (~16 row vectors in flight)
  const int lane = lane_id();
  const int VPR = a.H >> 3;
  const int total = nt * VPR;
  for (int v0 = lane; v0 < total; v0 += P * WAVE) {
    int tt[P], cc[P];
    float acc[P][8];
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int v = v0 + i * WAVE;
      tt[i] = v < total ? v / VPR : -1;
      cc[i] = v < total ? v - tt[i] * VPR : 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[i][e] = 0.0f;
    }
    u32x4_t o[P][KS];
    float w[P][KS];
#pragma unroll
    for (int i = 0; i < P; ++i)
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        const int s = tt[i] >= 0 ? sl[tt[i] * KS + j] : -1;
        w[i][j] = s >= 0 ? wt[tt[i] * KS + j] : 0.0f;
        o[i][j] = *reinterpret_cast<const u32x4_t*>((s >= 0 ? a.O + (size_t)s * a.H : a.x) + cc[i] * 8);
      }
#pragma unroll
    for (int i = 0; i < P; ++i)
#pragma unroll
      for (int j = 0; j < KS; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[i][2 * q] += w[i][j] * bf16_lo(o[i][j][q]);
          acc[i][2 * q + 1] += w[i][j] * bf16_hi(o[i][j][q]);
        }
#pragma unroll
    for (int i = 0; i < P; ++i) {
      if (tt[i] < 0) continue;
      u32x4_t r;
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = pack_bf16x2(acc[i][2 * q], acc[i][2 * q + 1]);
      __builtin_nontemporal_store(r, reinterpret_cast<u32x4_t*>(a.y + (size_t)(g0 + tt[i]) * a.H + cc[i] * 8));
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
}

// A wavefront combines tokens [g0, g0 + nt).  In the megakernel (S given) it
// first waits until every GEMM1 column tile of each row tile holding one of
// those tokens' source rows is done: every lane with a source row polls its
// row tile's counter, all in one vector load per round.
// Returns false when the launch was aborted.  With tracing on, t_ready gets
// the time the waits ended.
__device__ __forceinline__ bool combine_tokens(const FwdArgs& a, const Sched* S, Scratch& W, int g0, int nt,
                                               uint64_t& t_ready) {
  const int lane = lane_id();
  int* sl = W.wsl[wave_id()];
  float* wt = W.wwt[wave_id()];
  const int k = a.k, ks = a.k + a.S;
  // source rows of token g0 + lane / ks, entry lane % ks
  int s = -1, id = -1;
  float w = 1.0f;
  if (lane < nt * ks) {
    const int t = lane / ks, j = lane - t * ks, g = g0 + t;
    int seg = -1;
    if (j < k) {
      s = a.slot[(size_t)g * k + j];
      w = a.topk_w[(size_t)g * k + j];
      if (s >= 0) {
        seg = a.topk_idx[(size_t)g * k + j] - a.e0;
        s = pair_row(a, S, g, seg, s);
      }
    } else if (g < a.Tr) {
      seg = a.El + (j - k);
      s = shared_row(a, S, g, j - k);
    }
    if (S && s >= 0) {
      // row tile of the source row: its segment's first row tile plus its
      // place in the segment
      const int v = (int)(((long long)g * S->K) / a.T) * S->nseg + seg;
      id = S->mb[v] + (s - S->row0[v]) / BM;
      if ((unsigned)id >= (unsigned)a.mt_max) id = -1;
    }
  }
  // compact each token's present source rows, keeping their order: token t's
  // r-th present row goes to entry t * kp + r, kp being the most any token of
  // the unit has, so the passes below keep ~16 present rows in flight per
  // lane however sparse the local slots are (absent rows add nothing, so the
  // sum is unchanged)
  const uint64_t pm = __builtin_amdgcn_ballot_w64(s >= 0);
  const uint64_t tok = (1ull << ks) - 1;  // ks <= 16
  int kp = 0;
  for (int t = 0; t < nt; ++t) kp = max(kp, (int)__builtin_popcountll(pm & (tok << (t * ks))));
  sl[lane] = -1;
  __builtin_amdgcn_wave_barrier();
  if (s >= 0) {
    const int t = lane / ks;
    const int r = (int)__builtin_popcountll(pm & ((1ull << lane) - 1) & (tok << (t * ks)));
    sl[t * kp + r] = s;
    wt[t * kp + r] = w;
  }
  if (S) {
    // every column tile of the row tile (split ones reduced)
    if (!wave_wait_all(a, id >= 0 ? &a.ctl[CTL_READY + (2 * a.mt_max + id) * CTL_PAD] : nullptr, a.nt1)) return false;
    if (a.trace) t_ready = now_ticks();
  }
  __builtin_amdgcn_wave_barrier();
  switch (kp) {
#define MOE_COMBINE_CASE(n) \
  case n: combine_body<n>(a, sl, wt, g0, nt); break;
    case 0:  // no token of the unit has a source row: zero rows
    MOE_COMBINE_CASE(1) MOE_COMBINE_CASE(2) MOE_COMBINE_CASE(3) MOE_COMBINE_CASE(4)
    MOE_COMBINE_CASE(5) MOE_COMBINE_CASE(6) MOE_COMBINE_CASE(7) MOE_COMBINE_CASE(8)
    MOE_COMBINE_CASE(9) MOE_COMBINE_CASE(10) MOE_COMBINE_CASE(11) MOE_COMBINE_CASE(12)
    MOE_COMBINE_CASE(13) MOE_COMBINE_CASE(14) MOE_COMBINE_CASE(15) MOE_COMBINE_CASE(16)
#undef MOE_COMBINE_CASE
    default: break;
  }
  __builtin_amdgcn_wave_barrier();
  return true;
}

// ===========================================================================
// Compute work: one tile of GEMM0 (+SiLU*up) or one split of a GEMM1 tile.
// ===========================================================================
struct TileRef {
  int q, ph, seg, mt, nt, ks, rows;
};

// tile code: stage << 24 | class << 21 | index in the class queue.  A class
// queue holds its stage's tiles by readiness level, then segment, then slab,
// then row tile: the first claims go to the row tiles whose inputs are
// complete first, and the tiles of one level share their weight slabs.
__device__ __forceinline__ TileRef decode_tile(const FwdArgs& a, const Sched& S, int code) {
  const int stage = code >> 24, x = (code >> 21) & (NXCD - 1);
  int i = code & ((1 << 21) - 1);
  TileRef r;
  const int qp = stage_qph(stage, S.K);
  r.q = qp >> 1;
  r.ph = qp & 1;
  const int nsx = class_slabs(phase_slabs(a, r.ph), x);
  const int* cum = S.lvl[r.q];
  int L = 0;
  while (L < NLVL && i >= nsx * cum[L]) ++L;
  if (L > 0) i -= nsx * cum[L - 1];
  int seg = 0, rows = 0, c = 1, lo = 0;
  for (; seg < S.nseg; ++seg) {
    rows = S.rows[r.q * S.nseg + seg];
    const bool sh = seg >= a.El;
    c = level_tiles(rows, sh, L);
    if (i < nsx * c) {
      lo = level_lo(rows, sh, L);
      break;
    }
    i -= nsx * c;
  }
  r.seg = seg;
  r.mt = lo + i % c;
  const int slab = x + NXCD * (i / c);
  if (r.ph == 0) {
    r.nt = slab;
    r.ks = 0;
  } else {
    r.nt = slab / a.nsplit;
    r.ks = slab % a.nsplit;
  }
  r.rows = min(BM, rows - r.mt * BM);
  return r;
}

// Claims the next tile for a workgroup on XCD `home` (thread 0): its own
// class of the current stage first, then the other classes of that stage;
// the next stage only once every class of this one is exhausted, so a GEMM1
// tile is taken only when every GEMM0 tile of its chunk has been claimed by a
// running workgroup.  ph_only >= 0 restricts to one phase.  Returns the tile
// code or -1.
__device__ __forceinline__ int claim_tile(const FwdArgs& a, const Sched& S, int base, int ph_only, int home,
                                          int& stage, uint32_t& exhausted) {
  for (; stage < 2 * S.K; ++stage, exhausted = 0u) {
    if (ph_only >= 0 && (stage_qph(stage, S.K) & 1) != ph_only) continue;
    for (int j = 0; j < NXCD; ++j) {
      const int x = (home + j) & (NXCD - 1);
      const int n = S.ncls[stage][x];
      if (n == 0 || ((exhausted >> x) & 1u)) continue;
      int* q = &a.ctl[base + (stage * NXCD + x) * CTL_PAD];
      // other classes are read first so that exhausted queues take no atomic
      if (j > 0 && ld_relaxed(q) >= n) { exhausted |= 1u << x; continue; }
      const int i = fetch_add_relaxed(q, 1);
      if (i < n) return (stage << 24) | (x << 21) | i;
      exhausted |= 1u << x;
    }
  }
  return -1;
}

// Runs one GEMM0 tile or one split of a GEMM1 tile.  One mainloop instance
// serves both GEMMs; only the operands and the epilogue differ.
// Thread 0 claims the next tile (claim_next) between the mainloop and the
// epilogue (returned on thread 0), so the claim's round trip overlaps the
// epilogue stores.
template <int CP, typename ClaimFn>
__device__ __forceinline__ int run_gemm(const FwdArgs& a, const Sched& S, const TileRef& r, char* ring,
                                        ClaimFn&& claim_next) {
  const int qs = r.q * S.nseg + r.seg;
  const size_t orow = (size_t)S.row0[qs] + (size_t)r.mt * BM;
  const int n0 = r.nt * BN;
  // A: the dispatched rows and h are group-tiled (gemm::AOp); a shared
  // expert reads the caller's row-major x.  B: slab r.nt of the expert's
  // slab-tiled weights (n0 is a multiple of the slab height, so the slab
  // starts at element n0 * K), then the split's first k-step block.
  gemm::AOp A;
  const uint16_t* Bop;
  int Kd;
  A.rows = r.rows;
  if (r.ph == 0) {
    const size_t arow = (size_t)S.arow0[qs] + (size_t)r.mt * BM;
    if (r.seg < a.El) {
      A = {a.A + (arow >> 5) * (size_t)a.H * gemm::GROUP, a.H, (int)(arow & 31), a.H * gemm::GROUP * 2, r.rows};
    } else {
      A = {a.x + arow * a.H, a.H, 0, 0, r.rows};
    }
    Bop = a.w13 + (size_t)r.seg * slab_rows(2 * a.F) * a.H + (size_t)n0 * a.H;
    Kd = a.H;
  } else {
    const int kl = a.F / a.nsplit;
    A = {a.Hb + (orow >> 5) * (size_t)a.F * gemm::GROUP + (size_t)r.ks * kl * gemm::GROUP, a.F, (int)(orow & 31),
         a.F * gemm::GROUP * 2, r.rows};
    Bop = a.w2t + (size_t)r.seg * slab_rows(a.H) * a.F + (size_t)n0 * a.F + (size_t)r.ks * kl * SLAB;
    Kd = kl;
  }
  gemm::Acc acc;
  gemm::zero(acc);
  gemm::mainloop(acc, A, Bop, Kd, ring);
  int nxt = -1;
  if (threadIdx.x == 0) nxt = claim_next();
  if (r.ph == 0) {
    gemm::store_silu_mul_tiled_lds<CP>(acc, a.Hb + (orow >> 5) * (size_t)a.F * gemm::GROUP + (size_t)(n0 / 2) * gemm::GROUP,
                                       (int)(orow & 31), a.F * gemm::GROUP, r.rows, a.F - n0 / 2, ring);
  } else if (a.nsplit == 1) {
    gemm::store_bf16_lds<CP>(acc, a.O + orow * a.H + n0, a.H, r.rows, a.H - n0, ring);
  } else {
    gemm::store_f32<CP>(acc, a.part + ((size_t)r.ks * a.prow + orow) * a.H + n0, a.H, r.rows, a.H - n0);
  }
  return nxt;
}

// Split-K reduction of one GEMM1 tile by its last-arriving split: O rows
// [orow, orow + rows) x columns [n0, n0 + cols) = bf16(P_0 + P_1 + ... ) in
// split order, 4 columns per thread and step.  NS (the split count) is a
// template constant so that the loads of every split of a batch are issued
// before the first add: one memory round trip per batch.
template <int CP, int NS>
__device__ __forceinline__ void reduce_split_n(const FwdArgs& a, size_t orow, int rows, int n0, int cols) {
  const __amdgpu_buffer_rsrc_t rO = __builtin_amdgcn_make_buffer_rsrc(a.O, 0, -1, 0x00020000);
  const int q4 = cols >> 2;  // cols % 64 == 0
  const int total = rows * q4;
  const size_t pstride = (size_t)a.prow * a.H;
  constexpr int RB = NS >= 8 ? 4 : 32 / NS;  // 32 vectors in flight per thread
  for (int v0 = threadIdx.x; v0 < total; v0 += RB * FNTH) {
    f32x4_t u[RB][NS];
    // straight-line loads (a position past the tile re-reads the last one)
    // and one drain before the stores, so that every load is in flight at
    // once (see combine_body)
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int v = min(v0 + i * FNTH, total - 1);
      const int r = v / q4, c = (v - r * q4) * 4;
      const float* src = a.part + (orow + r) * (size_t)a.H + n0 + c;
#pragma unroll
      for (int p = 0; p < NS; ++p) u[i][p] = *reinterpret_cast<const f32x4_t*>(src + p * pstride);
    }
    gemm::wait_vm<0>();
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int v = v0 + i * FNTH;
      if (v >= total) continue;
      const int r = v / q4, c = (v - r * q4) * 4;
      f32x4_t t = u[i][0];
#pragma unroll
      for (int p = 1; p < NS; ++p)
#pragma unroll
        for (int j = 0; j < 4; ++j) t[j] += u[i][p][j];
      const size_t e = (orow + r) * (size_t)a.H + n0 + c;
      typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
      const u32x2_t packed = {pack_bf16x2(t[0], t[1]), pack_bf16x2(t[2], t[3])};
      if constexpr (CP == gemm::CP_PLAIN) *reinterpret_cast<u32x2_t*>(a.O + e) = packed;
      else __builtin_amdgcn_raw_buffer_store_b64(packed, rO, (uint32_t)(e * 2), 0, CP);
    }
  }
}

template <int CP>
__device__ __forceinline__ void reduce_split(const FwdArgs& a, size_t orow, int rows, int n0, int cols) {
  switch (a.nsplit) {
    case 2: reduce_split_n<CP, 2>(a, orow, rows, n0, cols); break;
    case 4: reduce_split_n<CP, 4>(a, orow, rows, n0, cols); break;
    case 8: reduce_split_n<CP, 8>(a, orow, rows, n0, cols); break;
    default: break;
  }
}

// After a GEMM1 item's partial stores have completed (all threads, past a
// barrier): counts its arrival; the last split of the tile reduces it.
// Returns true on the workgroup that reduced (its O stores still draining).
template <int CP>
__device__ __forceinline__ bool arrive_and_reduce(const FwdArgs& a, const Sched& S, Scratch& W, const TileRef& r,
                                                  int id) {
  if (threadIdx.x == 0)
    W.bc[3] = fetch_add_relaxed(&a.ctl[CTL_READY + (3 * a.mt_max + id * a.nt1 + r.nt) * CTL_PAD], 1);
  __syncthreads();
  const bool last = W.bc[3] == a.nsplit - 1;
  __syncthreads();
  if (!last) return false;
  const size_t orow = (size_t)S.row0[r.q * S.nseg + r.seg] + (size_t)r.mt * BM;
  reduce_split<CP>(a, orow, r.rows, r.nt * BN, min(BN, a.H - r.nt * BN));
  return true;
}

// ===========================================================================
// Prologue: the routing-derived workload and the plan (sections 3.1-3.3),
// computed redundantly by every workgroup from a small read of the stats.
// ===========================================================================
// sub: the chunk sub-offset tables staged in LDS (see moe_megakernel); the
// calibration table is staged here, in the same round trip.
// Wavefront argmin of (t, i) (lanes with i < 0 hold no point): the smallest
// t, the lowest i among equal ones, with n carried along; lane 0 ends with
// the result.  DPP exchanges within each row of 16 lanes (xor 1, xor 2, then
// the half-row and row mirrors, each pairing the lanes of two disjoint halves),
// then the four rows' results through readlane.  The order of the minimum
// with its index tie-break is total, so the pairing order does not matter.
__device__ __forceinline__ void argmin_take(double& t, int& i, int& n, double t2, int i2, int n2) {
  if (i2 >= 0 && (i < 0 || t2 < t || (t2 == t && i2 < i))) {
    t = t2;
    i = i2;
    n = n2;
  }
}
template <int CTRL>
__device__ __forceinline__ void argmin_dpp_step(double& t, int& i, int& n) {
  const uint64_t b = (uint64_t)__builtin_bit_cast(uint64_t, t);
  const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)b, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(b >> 32), CTRL, 0xF, 0xF, false);
  const int i2 = __builtin_amdgcn_mov_dpp(i, CTRL, 0xF, 0xF, false);
  const int n2 = __builtin_amdgcn_mov_dpp(n, CTRL, 0xF, 0xF, false);
  const double t2 = __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
  argmin_take(t, i, n, t2, i2, n2);
}
__device__ __forceinline__ void wave_argmin(double& t, int& i, int& n) {
  argmin_dpp_step<0xB1>(t, i, n);   // quad_perm [1, 0, 3, 2]
  argmin_dpp_step<0x4E>(t, i, n);   // quad_perm [2, 3, 0, 1]
  argmin_dpp_step<0x141>(t, i, n);  // row_half_mirror
  argmin_dpp_step<0x140>(t, i, n);  // row_mirror
  const uint64_t b = (uint64_t)__builtin_bit_cast(uint64_t, t);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)b, 16 * r);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), 16 * r);
    const int i2 = __builtin_amdgcn_readlane(i, 16 * r);
    const int n2 = __builtin_amdgcn_readlane(n, 16 * r);
    argmin_take(t, i, n, __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo), i2, n2);
  }
}

// The cost model's plan on the first wavefront (all 64 lanes call; lane 0
// ends with it in p): Eq 15 at every grid point, one point per lane, with its
// steal count (Eq 11-14) alongside; Eq 16 by a wavefront argmin in the host
// model's order (c ascending, then K): the smallest T_total, the lowest grid
// index among equal ones, which is the first strict minimum of the host's
// scan.  W.cal and W.st hold the calibration table and the routing stats.
__device__ __forceinline__ void model_plan(const FwdArgs& a, const Scratch& W, moe_plan& p) {
  const int tid = threadIdx.x;
  double wc, wd, wb;
  cm_volumes(W.st, a.H, a.F, a.S * a.Tr, W.cal.literal, &wc, &wd, &wb);
  const int nk = W.cal.n_k, npt = W.cal.n_c * nk;
  double best = 0.0;
  int bi = -1;
  for (int i = tid; i < npt; i += WAVE) {
    const double t = cm_t_total(W.cal, i / nk, i - (i / nk) * nk, wc, wd, wb);
    if (bi < 0 || t < best) { best = t; bi = i; }
  }
  int ns = 0;
  if (bi >= 0) {
    long long nt_by_k[MOE_CALIB_MAX_K];
    for (int j = 0; j < nk; ++j) nt_by_k[j] = W.st[ST_NTK + kopt_index(W.cal.kk[j])];
    moe_plan q;
    cm_finish(W.cal, a.N, wc, wd, wb, nt_by_k, bi / nk, bi - (bi / nk) * nk, best, &q);
    ns = q.n_steal;
  }
  wave_argmin(best, bi, ns);
  if (tid == 0) {
    p.c = W.cal.c[bi / nk];
    p.K = W.cal.kk[bi - (bi / nk) * nk];
    p.n_steal = ns;
    p.final_all = 1;
    p.t_pred_s = best;
  }
}

__device__ __forceinline__ void prologue_plan(const FwdArgs& a, Sched& S, Scratch& W) {
  const int tid = threadIdx.x;
  StoredPlan sp{};  // thread 0: the stored plan, read in the same round trip
  {
    // one memory round trip for the calibration table, the routing stats
    // and the schedule image for K = 1 (the usual pick; another K is loaded
    // once the plan has chosen it): every load is issued before the first
    // store to LDS
    constexpr int NCW = (int)(sizeof(DevCalib) / 4);
    constexpr int NC = (NCW + FNTH - 1) / FNTH;
    constexpr int NIV = (SCHED_WORDS - SCHED_IMG0) / 4;
    constexpr int NI = (NIV + FNTH - 1) / FNTH;
    const uint32_t* csrc = reinterpret_cast<const uint32_t*>(a.calib);
    const u32x4_t* isrc = reinterpret_cast<const u32x4_t*>(a.sched + SCHED_IMG0);
    uint32_t cv[NC];
    u32x4_t iv[NI];
    int sv = 0;
#pragma unroll
    for (int j = 0; j < NC; ++j) cv[j] = tid + j * FNTH < NCW ? csrc[tid + j * FNTH] : 0u;
    if (tid >= FNTH - ST_WORDS) sv = a.stats[tid - (FNTH - ST_WORDS)];
    if (tid == 0) sp = *stored_plan(a);
#pragma unroll
    for (int j = 0; j < NI; ++j)
      if (tid + j * FNTH < NIV) iv[j] = isrc[tid + j * FNTH];
    uint32_t* cdst = reinterpret_cast<uint32_t*>(&W.cal);
#pragma unroll
    for (int j = 0; j < NC; ++j)
      if (tid + j * FNTH < NCW) cdst[tid + j * FNTH] = cv[j];
    if (tid >= FNTH - ST_WORDS) W.st[tid - (FNTH - ST_WORDS)] = sv;
    if (tid == 0) W.bc[6] = sp.gen == a.calib_gen ? 1 : 0;
    u32x4_t* idst = reinterpret_cast<u32x4_t*>(reinterpret_cast<int*>(&S) + SCHED_IMG0);
#pragma unroll
    for (int j = 0; j < NI; ++j)
      if (tid + j * FNTH < NIV) idst[tid + j * FNTH] = iv[j];
  }
  __syncthreads();
  const bool model = !a.forced && a.mode != MOE_MODE_STATIC;
  moe_plan p;
  // the plan the routing's last kernel evaluated on these tables, when the
  // calibration has not changed since (W.bc[6]); else evaluated here
  if (model && !W.bc[6] && tid < WAVE) model_plan(a, W, p);
  if (tid == 0) {
    if (model && W.bc[6]) {
      p = sp.p;
    } else if (a.forced) {
      p = a.fplan;
    } else if (a.mode == MOE_MODE_STATIC) {
      p.c = W.cal.static_c;
      p.K = 1;
      p.n_steal = 0;
      p.final_all = 0;
      p.t_pred_s = 0.0;
    }
    S.c = p.c;
    W.bc[5] = p.K;
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
// store it with agent-coherent (sc1) stores and drain them before their
// relaxed increment, and no CU loads a line of a dispatched row, an Hbuf/O
// row or a partial before its counter says it is complete (the row map keeps
// every row tile's lines its own; the combine's absent entries read x), so no
// stale copy of those lines can sit in the consumer's L1 or L2 (caches are
// invalidated at kernel start).
// One lane polls *p until it reaches target, backing off exponentially up to
// about 0.85 us between reads (many waiters poll the same few lines); the
// abort word and the deadline are checked every eighth read.  Returns false
// on abort or timeout.
__device__ __forceinline__ bool poll_geq(const FwdArgs& a, const int* p, int target) {
  if (ld_relaxed(p) >= target) return true;
  const uint64_t deadline = now_ticks() + (uint64_t)a.timeout_ticks;
  int backoff = 1;
  for (int it = 1;; ++it) {
    for (int i = 0; i < backoff; ++i) __builtin_amdgcn_s_sleep(4);
    if (ld_relaxed(p) >= target) return true;
    backoff = min(backoff * 2, 8);
    if ((it & 7) == 0) {
      if (ld_relaxed(&a.ctl[CTL_ABORT])) return false;
      if (now_ticks() > deadline) {
        st_relaxed(&a.ctl[CTL_ABORT], 1);
        atomicOr(a.err, ERR_TIMEOUT);
        return false;
      }
    }
  }
}

__device__ __forceinline__ bool wait_geq(const FwdArgs& a, Scratch& W, const int* p, int target) {
  if (a.inject_stall) target += 1 << 30;
  if (threadIdx.x == 0) W.bc[2] = poll_geq(a, p, target) ? 1 : 0;
  __syncthreads();
  const int ok = W.bc[2];
  __syncthreads();
  return ok != 0;
}

// A compute worker whose GEMM0 row tile is not dispatched yet moves rows
// itself instead of idling (movement stealing, the mirror image of the
// section 3.2.2 bubble stealing): each wavefront claims and copies one
// dispatch unit, then the workgroup checks the counter again.  Once every
// unit is claimed it polls.
__device__ __forceinline__ bool wait_rows(const FwdArgs& a, const Sched& S, Scratch& W, const int* p, int target) {
  if (a.inject_stall) target += 1 << 30;
  const uint64_t deadline = now_ticks() + (uint64_t)a.timeout_ticks;
  for (;;) {
    if (threadIdx.x == 0) {
      int st = ld_relaxed(p) >= target ? 1 : 0;
      if (!st && (W.dexh || !a.move_steal)) st = poll_geq(a, p, target) ? 1 : -1;
      else if (!st && (ld_relaxed(&a.ctl[CTL_ABORT]) || now_ticks() > deadline)) {
        st_relaxed(&a.ctl[CTL_ABORT], 1);
        atomicOr(a.err, ERR_TIMEOUT);
        st = -1;
      }
      W.bc[2] = st;
    }
    __syncthreads();
    const int st = W.bc[2];
    __syncthreads();
    if (st) return st > 0;
    int shard = first_shard(W);
    const int u = claim_disp(a, S, shard);
    if (u >= 0) dispatch_one<true>(a, &S, W, u, unit_row(a, &S, u));
    else if (lane_id() == 0) W.dexh = 1;
  }
}

// Runs up to max_tiles compute tiles from the shared queue (all of them for a
// compute worker, n_steal for a movement worker).  A tile waits for its inputs
// (GEMM0: its rows dispatched; GEMM1: every GEMM0 column tile of its row
// tile), runs, and is published once every thread's agent-coherent output
// stores have completed, with one relaxed increment.  The next tile is claimed
// between mainloop and epilogue.  Returns false when the launch was aborted.
__device__ __forceinline__ bool compute_tiles(const FwdArgs& a, const Sched& S, Scratch& W, char* ring, int ticket,
                                              int max_tiles) {
  if (max_tiles <= 0) return true;
  const int home = xcd_id() & (NXCD - 1);
  int stage = 0;           // thread 0's claim position
  uint32_t exhausted = 0;  // classes of that stage found empty
  if (threadIdx.x == 0) W.bc[1] = claim_tile(a, S, a.qx, -1, home, stage, exhausted);
  __syncthreads();
  int t = __builtin_amdgcn_readfirstlane(W.bc[1]);
  __syncthreads();
  for (int done = 1; t >= 0; ++done) {
    jitter(a, 0x40000u + (uint32_t)t);
    const uint64_t t0 = a.trace ? now_ticks() : 0;
    const TileRef r = decode_tile(a, S, t);
    const int id = S.mb[r.q * S.nseg + r.seg] + r.mt;
    if (r.ph == 0) {
      if (r.seg < a.El && !wait_rows(a, S, W, &a.ctl[CTL_READY + id * CTL_PAD], r.rows)) return false;
    } else {
      if (!wait_geq(a, W, &a.ctl[CTL_READY + (a.mt_max + id) * CTL_PAD], a.nt0)) return false;
    }
    const uint64_t t1 = a.trace ? now_ticks() : 0;
    const bool more = done < max_tiles;
    const int nxt = run_gemm<gemm::CP_SC1>(a, S, r, ring, [&] { return more ? claim_tile(a, S, a.qx, -1, home, stage, exhausted) : -1; });
    __builtin_amdgcn_s_waitcnt(0);
    if (threadIdx.x == 0) W.bc[1] = nxt;
    __syncthreads();  // every thread's output stores have completed
    // GEMM0 tile: its row tile gains a column; GEMM1 tile (or the last split
    // of one, after it reduced the tile): its row tile gains a column
    bool publish = true;
    if (r.ph == 1 && a.nsplit > 1) {
      publish = arrive_and_reduce<gemm::CP_SC1>(a, S, W, r, id);
      if (publish) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
      }
    }
    if (threadIdx.x == 0) {
      if (publish) fetch_add_relaxed(&a.ctl[CTL_READY + ((r.ph == 0 ? 1 : 2) * a.mt_max + id) * CTL_PAD], 1);
      if (a.trace) trace_rec(a, W, 2, ticket, t, t0, t1, now_ticks());
    }
    t = __builtin_amdgcn_readfirstlane(W.bc[1]);  // rewritten only after the next mainloop's barriers
  }
  return true;
}

// wavefront-level wait on up to 64 counters at once: each lane with p set
// waits for *p >= target, one vector load per round for all of them
__device__ __forceinline__ bool wave_wait_all(const FwdArgs& a, const int* p, int target) {
  if (a.inject_stall) target += 1 << 30;
  bool done = p == nullptr || ld_relaxed(p) >= target;
  if (__builtin_amdgcn_ballot_w64(!done) == 0) return true;
  const uint64_t deadline = now_ticks() + (uint64_t)a.timeout_ticks;
  int backoff = 1;
  for (int it = 1;; ++it) {
    for (int i = 0; i < backoff; ++i) __builtin_amdgcn_s_sleep(4);
    if (!done) done = ld_relaxed(p) >= target;
    if (__builtin_amdgcn_ballot_w64(!done) == 0) return true;
    backoff = min(backoff * 2, 8);
    if ((it & 7) == 0) {
      int stop = 0;
      if (lane_id() == 0) {
        if (ld_relaxed(&a.ctl[CTL_ABORT])) {
          stop = 1;
        } else if (now_ticks() > deadline) {
          st_relaxed(&a.ctl[CTL_ABORT], 1);
          atomicOr(a.err, ERR_TIMEOUT);
          stop = 1;
        }
      }
      if (__builtin_amdgcn_readfirstlane(stop)) return false;
    }
  }
}

// Combine units (ct tokens, in token and hence chunk order) are claimed per
// wavefront from the sharded combine queue until every unit is claimed; each
// waits only for the row tiles its tokens' rows come from, so the combine of
// finished tokens starts while the last GEMM tiles run.
__device__ __forceinline__ bool combine_claimed(const FwdArgs& a, const Sched& S, Scratch& W, int ticket) {
  // at most one wavefront per unit joins, the lowest arrival tickets first
  // (movement workers before compute workers): with fewer units than
  // wavefronts the others' claims could only fail, on the same few counters
  if (ticket * NWF + wave_id() >= S.n_comb) return true;
  int shard = first_shard(W);
  for (;;) {
    const int u = claim_unit(a, CTL_QC, S.n_comb, shard);
    if (u < 0) return true;
    jitter(a, 0x10000u + (uint32_t)u);
    const uint64_t t0 = a.trace ? now_ticks() : 0;
    uint64_t t1 = t0;
    const int g0 = u * a.ct;
    if (!combine_tokens(a, &S, W, g0, min(a.ct, a.T - g0), t1)) return false;
    if (a.trace && lane_id() == 0) trace_rec(a, W, 4, ticket, u | ((long long)wave_id() << 24), t0, t1, now_ticks());
  }
}

// ===========================================================================
// The persistent megakernel: one workgroup per CU, all resident at once (the
// host checks that the GPU holds N of them).  The first c workgroups to
// arrive become movement workers.  Every wait ends at the abort word or the
// timeout, so workers that cannot start (the CUs held by other work) turn
// into MOE_ERR_TIMEOUT, never a hang.
// ===========================================================================
// One layer, run by this workgroup.  next: the following layer of a
// stacked launch, whose dispatch the movement workers start.
__device__ __forceinline__ void mega_layer(const FwdArgs& a, Sched& S, Scratch& W, char* ring, const FwdArgs* next) {
  const int tid = threadIdx.x;
  const uint64_t t_entry = a.trace ? now_ticks() : 0;

  if (blockIdx.x == 0)
    for (int i = tid; i < a.ctl_words; i += FNTH) a.ctl_next[i] = 0;

  // arrival ticket (role) first, so that its round trip overlaps the staging
  jitter(a, 0);
  int tk = 0;
  if (tid == 0) {
    tk = fetch_add_relaxed(&a.ctl[CTL_TICKET], 1);
    W.dexh = 0;
  }

  prologue_plan(a, S, W);
  if (W.bc[5] != 1) load_sched(a, S, W.bc[5]);  // K = 1's image came with the calibration

  if (tid < NWF) W.tcnt[tid] = 0;
  if (tid == 0) {
    // the ticket's round trip overlapped the plan
    W.bc[0] = tk;
    W.ticket = tk;
    S.disp0 = a.static_disp ? (a.move_steal ? ceil_div(S.bnd[1], a.dt) : min(S.n_disp, S.c * NWF)) : 0;
  }
  __syncthreads();
  const int ticket = __builtin_amdgcn_readfirstlane(W.bc[0]);
  const bool mover = ticket < S.c;
  const uint64_t t_sched = a.trace ? now_ticks() : 0;
  __syncthreads();

  // this wavefront's statically owned dispatch units, if any: with movement
  // stealing every unit of the first chunk, round-robin over all wavefronts
  // (that chunk's dispatch at the full chip's copy rate before the first
  // tile, whose rows would otherwise wait for units claimed one by one; the
  // later chunks' units go through the queue, beside the first chunk's
  // GEMMs); else one unit per wavefront of the movement workers
  {
    const int stride = (a.move_steal ? (int)gridDim.x : S.c) * NWF;
    for (int u0 = ticket * NWF + wave_id(); u0 < S.disp0; u0 += stride)
      dispatch_one<true>(a, &S, W, u0, unit_row(a, &S, u0));
  }

  bool ok = true;
  if (mover) {
    // dispatch: every token row, in token (hence chunk) order
    dispatch_claimed(a, S, W);
    __syncthreads();
    if (a.trace && tid == 0) trace_rec(a, W, 3, ticket, 0, t_sched, now_ticks(), 0);
    // the next layer's dispatch beside this layer's GEMMs
    if (next) dispatch_ahead(*next, W);
    // bubble stealing: n_steal GEMM tiles right after dispatch (section 3.2.2)
    ok = compute_tiles(a, S, W, ring, ticket, S.n_steal);
    if (ok) combine_claimed(a, S, W, ticket);
  } else {
    ok = compute_tiles(a, S, W, ring, ticket, 1 << 30);
    // the final combine on every worker (section 4): once the compute queue
    // is empty a compute worker joins the combine; in a stacked launch with a
    // layer after this one it goes on to that layer's GEMMs instead, and this
    // layer's movement workers combine meanwhile (on a few CUs a copy moves
    // more bytes per CU than on all of them)
    if (ok && S.final_all && !a.stack_next) combine_claimed(a, S, W, ticket);
  }
  if (a.trace) {
    __syncthreads();
    if (tid == 0) trace_rec(a, W, 1, ticket, mover ? 1 : 0, t_entry, t_sched, now_ticks());
    __syncthreads();
    // each wavefront's record count, and (block 0) the header
    int* hdr = reinterpret_cast<int*>(a.trace);
    if (tid < NWF) hdr[TRACE_HDR / 4 + blockIdx.x * NWF + tid] = min(W.tcnt[tid], a.trace_cap);
    if (blockIdx.x == 0 && tid == 0) {
      hdr[1] = (int)gridDim.x * NWF;
      hdr[2] = a.trace_cap;
      hdr[3] = a.trace_rec0;
      hdr[0] = TRACE_MAGIC;
    }
  }
}

__global__ void __launch_bounds__(FNTH, 1) moe_megakernel(FwdArgs a) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(1024))) char ring[gemm::RING_BYTES];
  mega_layer(a, S, W, ring, nullptr);
}

// Several independent layers (they share x, not their outputs) in one
// persistent launch: a workgroup moves on to layer l + 1 as soon as it finds
// no more work to claim in layer l, so layer l + 1's dispatch and first GEMM
// tiles run while layer l's last tiles and its combine finish.  Every item of
// layer l is claimed by a workgroup still in layer l, and no wait depends on
// a later layer, so every wait ends.
// The layers' argument blocks are read in place from the kernel argument
// segment (constant memory, scalar loads): indexing the by-value parameter
// with the layer number would copy it to scratch.
__global__ void __launch_bounds__(FNTH, 1) moe_megakernel_stack(StackArgs st) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(1024))) char ring[gemm::RING_BYTES];
  (void)st;
  const __attribute__((address_space(4))) StackArgs* ka =
      (const __attribute__((address_space(4))) StackArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  const int n = ka->n;
  for (int l = 0; l < n; ++l) {
    __syncthreads();  // the previous layer's LDS state is dead
    mega_layer(*(const FwdArgs*)&ka->layer[l], S, W, ring, l + 1 < n ? (const FwdArgs*)&ka->layer[l + 1] : nullptr);
  }
}

// ===========================================================================
// Serial baseline: four kernels, each on every CU, no overlap.
// ===========================================================================
// The schedule images of the routing tables just built: workgroup ki builds
// the schedule for K = 2^ki in LDS and stores it.
__global__ void __launch_bounds__(FNTH, 1) sched_build_kernel(FwdArgs a) {
  __shared__ Sched S;
  __shared__ Scratch W;
  const int ki = blockIdx.x;
  build_sched(a, a.sub_off, a.row_off, S, W, 1 << ki);
  const int* src = reinterpret_cast<const int*>(&S);
  int32_t* dst = const_cast<int32_t*>(a.sched) + (size_t)ki * SCHED_WORDS;  // the images' one writer
  for (int i = SCHED_IMG0 + threadIdx.x; i < SCHED_WORDS; i += FNTH) dst[i] = src[i];
  if (ki != 0) return;
  // the cost model's plan of these tables under the current calibration
  // (every workgroup of a launch would evaluate the same; a prologue whose
  // calibration generation differs evaluates it again)
  const uint32_t* csrc = reinterpret_cast<const uint32_t*>(a.calib);
  uint32_t* cdst = reinterpret_cast<uint32_t*>(&W.cal);
  for (int i = threadIdx.x; i < (int)(sizeof(DevCalib) / 4); i += FNTH) cdst[i] = csrc[i];
  for (int i = threadIdx.x; i < ST_WORDS; i += FNTH) W.st[i] = a.stats[i];
  __syncthreads();
  moe_plan p;
  if (threadIdx.x < WAVE) model_plan(a, W, p);
  if (threadIdx.x == 0) {
    StoredPlan* sp = const_cast<StoredPlan*>(stored_plan(a));
    sp->p = p;
    sp->gen = a.calib_gen;
  }
}

__global__ void __launch_bounds__(FNTH, 1) serial_dispatch_kernel(FwdArgs a) {
  __shared__ Scratch W;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0)
    for (int i = tid; i < a.ctl_words; i += FNTH) a.ctl_next[i] = 0;
  dispatch_static(a, W, blockIdx.x * NWF + wave_id(), gridDim.x * NWF);
}

template <int PH>
__device__ __forceinline__ void serial_gemm(const FwdArgs& a) {
  __shared__ Sched S;
  __shared__ Scratch W;
  __shared__ __attribute__((aligned(1024))) char ring[gemm::RING_BYTES];
  load_sched(a, S, a.serial_K);
  const int home = xcd_id() & (NXCD - 1);
  int stage = 0;
  uint32_t exhausted = 0;
  if (threadIdx.x == 0) W.bc[1] = claim_tile(a, S, a.qxs, PH, home, stage, exhausted);
  __syncthreads();
  int t = __builtin_amdgcn_readfirstlane(W.bc[1]);
  __syncthreads();
  while (t >= 0) {
    const TileRef r = decode_tile(a, S, t);
    const bool split = PH == 1 && a.nsplit > 1;
    auto next = [&] { return claim_tile(a, S, a.qxs, PH, home, stage, exhausted); };
    // split partials are read by another workgroup within this kernel:
    // agent-coherent stores, drained before the arrival count
    const int nxt = split ? run_gemm<gemm::CP_SC1>(a, S, r, ring, next) : run_gemm<gemm::CP_PLAIN>(a, S, r, ring, next);
    if (split) __builtin_amdgcn_s_waitcnt(0);
    if (threadIdx.x == 0) W.bc[1] = nxt;
    __syncthreads();
    if (split) arrive_and_reduce<gemm::CP_PLAIN>(a, S, W, r, S.mb[r.q * S.nseg + r.seg] + r.mt);
    t = __builtin_amdgcn_readfirstlane(W.bc[1]);  // rewritten only after the next mainloop's barriers
  }
}

__global__ void __launch_bounds__(FNTH, 1) serial_gemm0_kernel(FwdArgs a) { serial_gemm<0>(a); }
__global__ void __launch_bounds__(FNTH, 1) serial_gemm1_kernel(FwdArgs a) { serial_gemm<1>(a); }

__global__ void __launch_bounds__(FNTH, 1) serial_combine_kernel(FwdArgs a) {
  __shared__ Scratch W;
  const int n = ceil_div(a.T, a.ct);
  for (int u = blockIdx.x * NWF + wave_id(); u < n; u += gridDim.x * NWF) {
    const int g0 = u * a.ct;
    uint64_t t_unused = 0;
    combine_tokens(a, nullptr, W, g0, min(a.ct, a.T - g0), t_unused);
  }
}

}  // namespace moe
