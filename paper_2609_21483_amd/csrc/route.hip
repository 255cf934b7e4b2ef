// Routing that precedes the MoE layer (the layer takes the routing result as
// its input, paper section 4) and the routing tables of this GPU's share
// (section 3.1 descriptors X_local, X_in, X_in^uniq; the dispatch permutation
// and its deduplication, section 4; the chunk offsets of section 3.2.1).
//
// Everything here is deterministic: the routing decisions are those of logits
// with one fp32 accumulator per (token, expert) over ascending h, and slots
// come from block histograms, an ordered scan and wavefront ballots, never
// from atomic slot claiming.
#include "common.h"
#include "gemm.h"
#include "kernels.h"

namespace moe {

// ---------------------------------------------------------------------------
// Gate: logits -> softmax -> top-k (on logits, ties -> smaller id) -> renormalise
//
// The logit of (token g, expert e) is defined in fp32 with one accumulator,
// hidden index ascending, each product rounded to fp32 before it is added,
// then + bias[e].  That sum is a chain of H dependent additions, so it is
// evaluated only where it can change the routing, and the selection is still
// exactly the one the full definition gives:
//   1. gate_prep:  WgT = Wg transposed ([E][H]) and ||w_e||_2.
//   2. gate_mfma:  approximate logits L~ by bf16 MFMA (fp32 accumulation) and
//                  ||x_g||_2.
//   3. gate_select: per token, a bound d_e >= |L - L~| (from the worst-case
//      error of the two summations, |x|.|w| <= ||x|| ||w||) gives intervals
//      [L~ - d, L~ + d] that hold the defined logits.  tau = k-th largest lower
//      end; every expert whose upper end reaches tau is a candidate.  The true
//      top-k lie among the candidates and every other expert is strictly
//      below the k-th logit, so the top-k of the candidates' exact logits
//      (the defined chains) is the top-k of all experts.
// Softmax weights come from the exact logits of the chosen experts; the
// normaliser over all experts cancels in the renormalisation up to rounding.
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(NTH) gate_prep_kernel(GateArgs a) {
  __shared__ float part[NTH / WAVE];
  const int e = blockIdx.x;
  const int tid = threadIdx.x;
  if (e == 0 && tid == 0) a.stats[ST_CANDS] = 0;  // the candidate pass counts the chains from here
  float ss = 0.0f;
  // PREP_V loads in flight per thread before their stores (the column of
  // Wg is strided by E, one 2-byte read per value)
  constexpr int PREP_V = 16;
  for (int h0 = 0; h0 < a.H; h0 += PREP_V * NTH) {
    uint16_t v[PREP_V];
#pragma unroll
    for (int i = 0; i < PREP_V; ++i) {
      const int h = h0 + i * NTH + tid;
      v[i] = h < a.H ? a.wg[(size_t)h * a.E + e] : (uint16_t)0;
    }
#pragma unroll
    for (int i = 0; i < PREP_V; ++i) {
      const int h = h0 + i * NTH + tid;
      if (h < a.H) {
        a.wgt[(size_t)e * a.H + h] = v[i];
        const float f = bf16_to_f32(v[i]);
        ss += f * f;
      }
    }
  }
#pragma unroll
  for (int d = WAVE / 2; d > 0; d >>= 1) ss += __shfl_xor(ss, d, WAVE);
  if ((tid & (WAVE - 1)) == 0) part[tid / WAVE] = ss;
  __syncthreads();
  if (tid == 0) {
    float t = 0.0f;
    for (int w = 0; w < NTH / WAVE; ++w) t += part[w];
    a.wn[e] = sqrtf(t);
  }
}

// 32 tokens x all experts per workgroup, v_mfma_f32_32x32x16_bf16 with the
// operands read straight from global memory.  Each of the 4 wavefronts sums
// a quarter of the hidden range (any order is allowed here: the bound below
// covers recursive fp32 summation of all H products) and the quarters are
// added through LDS.  Lane l holds token row (l & 31) and expert row (l & 31)
// of the current 32-expert block at hidden offsets 8 * (l >> 5) .. + 8 of each
// 16-deep step; GSTEP steps are loaded before their MFMAs.  GATE_EB 32-expert
// blocks are summed per pass over H: one block with 8 steps ahead when E <= 32
// (the pass streams x with more loads in flight), four with 4 steps ahead
// otherwise (register budget).
template <int GATE_EB, int GSTEP, int GWAVES>
__device__ __forceinline__ void gate_mfma_body(const GateArgs& a, float (*red)[32 * 32 * 4], float (*ssr)[64]) {
  const int lane = threadIdx.x & (WAVE - 1), wave = threadIdx.x / WAVE;
  const int g0 = blockIdx.x * 32;
  const int row = lane & 31, kh = (lane >> 5) * 8;
  const int g = g0 + row;
  const bool grow = g < a.T;
  const int hq = a.H / GWAVES;  // multiple of 16
  const int hbeg = wave * hq;
  const uint16_t* xr = a.x + (size_t)(grow ? g : 0) * a.H + kh + hbeg;
  float ss = 0.0f;
  for (int eb0 = 0; eb0 < a.E; eb0 += 32 * GATE_EB) {
    const int nb = min(GATE_EB, (a.E - eb0 + 31) / 32);
    f32x16_t acc[GATE_EB];
    const uint16_t* wr[GATE_EB];
    bool ev[GATE_EB];
#pragma unroll
    for (int b = 0; b < GATE_EB; ++b) {
      acc[b] = f32x16_t{};
      const int e = eb0 + 32 * b + row;
      ev[b] = e < a.E;
      wr[b] = a.wgt + (size_t)(ev[b] ? e : 0) * a.H + kh + hbeg;
    }
    // GSTEP steps of operands per set; the next set is loaded before the
    // MFMAs of the current one
    bf16x8_t xa[2][GSTEP], wb[2][GSTEP][GATE_EB];
    auto load_set = [&](int set, int h0) {
#pragma unroll
      for (int st = 0; st < GSTEP; ++st) {
        const int h = h0 + 16 * st;
        xa[set][st] = bf16x8_t{};
        if (h < hq && grow) xa[set][st] = *reinterpret_cast<const bf16x8_t*>(xr + h);
#pragma unroll
        for (int b = 0; b < GATE_EB; ++b) {
          wb[set][st][b] = bf16x8_t{};
          if (b < nb && h < hq && ev[b]) wb[set][st][b] = *reinterpret_cast<const bf16x8_t*>(wr[b] + h);
        }
      }
    };
    auto mfma_set = [&](int set) {
#pragma unroll
      for (int st = 0; st < GSTEP; ++st) {
        if (eb0 == 0) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float f = (float)xa[set][st][q];
            ss += f * f;
          }
        }
#pragma unroll
        for (int b = 0; b < GATE_EB; ++b)
          if (b < nb) acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[set][st], wb[set][st][b], acc[b], 0, 0, 0);
      }
    };
    load_set(0, 0);
    int h0 = 0;
    for (; h0 + 16 * GSTEP < hq; h0 += 32 * GSTEP) {
      load_set(1, h0 + 16 * GSTEP);
      mfma_set(0);
      if (h0 + 32 * GSTEP < hq) load_set(0, h0 + 32 * GSTEP);
      mfma_set(1);
    }
    if (h0 < hq) mfma_set(0);
    // add the quarters: C[8 (r >> 2) + 4 (l >> 5) + (r & 3)][l & 31]
    if (wave > 0) {
#pragma unroll
      for (int b = 0; b < GATE_EB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[wave - 1][(b * 16 + r) * WAVE + lane] = acc[b][r];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int b = 0; b < GATE_EB; ++b) {
        const int e = eb0 + 32 * b + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float v = acc[b][r];
#pragma unroll
          for (int w = 0; w < GWAVES - 1; ++w) v += red[w][(b * 16 + r) * WAVE + lane];
          const int gr = g0 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (b < nb && e < a.E && gr < a.T) a.lt[(size_t)gr * a.E + e] = v;
        }
      }
    }
    __syncthreads();
  }
  ssr[wave][lane] = ss;
  __syncthreads();
  if (wave == 0) {
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < GWAVES; ++w) t += ssr[w][lane] + ssr[w][lane ^ 32];
    if (lane < 32 && grow) a.xn[g] = sqrtf(t);
  }
}


// lanes of one token's group of GG: reductions stay inside the group
constexpr int GG = 16;
constexpr int GTOK = NTH / GG;    // tokens per workgroup

__device__ __forceinline__ bool better(float v, int e, float bv, int be) {
  return v > bv || (v == bv && e < be);
}
__device__ __forceinline__ void group_argmax(float& v, int& e) {
#pragma unroll
  for (int d = GG / 2; d > 0; d >>= 1) {
    const float ov = __shfl_xor(v, d, WAVE);
    const int oe = __shfl_xor(e, d, WAVE);
    if (better(ov, oe, v, e)) { v = ov; e = oe; }
  }
}

// approximate logit of (g, e) with bias, and its half-width
__device__ __forceinline__ void interval(const GateArgs& a, int g, int e, float xn, float& l, float& d) {
  l = a.lt[(size_t)g * a.E + e];
  if (a.bias) l = l + a.bias[e];
  d = a.bound * xn * a.wn[e];
  d = d + 4.0f * 5.9604645e-8f * (fabsf(l) + d) + 1e-30f;
}

// Candidates of the ntok tokens from g0 (one workgroup of NTH threads, GTOK
// tokens per pass, a token's experts spread over the GG lanes of its group,
// EPL each): tau = the k-th largest lower end; every expert whose upper end
// reaches tau becomes a chain (g, e) of the chain list.  A first pass counts
// each token's candidates, the tile takes its range of the list with one
// atomic, and a second pass writes each token's chains in ascending expert
// order (experts of neighbouring chains then differ in their low bits,
// which spreads the chain kernel's reads of their gate rows over the LDS
// banks).  t_cnt, t_off, t_tau: ntok entries of workgroup memory.
template <int EPL>
__device__ __forceinline__ void cand_tile(const GateArgs& a, int g0, int ntok, int* t_cnt, int* t_off, float* t_tau,
                                          int& base_s) {
  const int tid = threadIdx.x, grp = tid / GG, gl = tid % GG;
  for (int t0 = 0; t0 < ntok; t0 += GTOK) {
    const int g = g0 + t0 + grp;
    const bool valid = g < a.T;
    const int gs = valid ? g : 0;
    const float xn = a.xn[gs];
    float lo[EPL], hi[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = gl + GG * i;
      lo[i] = hi[i] = -INFINITY;
      if (e < a.E) {
        float l, d;
        interval(a, gs, e, xn, l, d);
        lo[i] = l - d;
        hi[i] = l + d;
      }
    }
    float tau = -INFINITY;
    for (int r = 0; r < a.k; ++r) {
      float v = -INFINITY;
      int e = 1 << 30;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (better(lo[i], gl + GG * i, v, e)) { v = lo[i]; e = gl + GG * i; }
      group_argmax(v, e);
      tau = v;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (gl + GG * i == e) lo[i] = -INFINITY;
    }
    int mine = 0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) mine += valid && hi[i] >= tau;
#pragma unroll
    for (int d = GG / 2; d > 0; d >>= 1) mine += __shfl_xor(mine, d, WAVE);
    if (gl == 0) {
      t_cnt[t0 + grp] = mine;
      t_tau[t0 + grp] = tau;
    }
  }
  __syncthreads();
  if (tid < WAVE) {  // exclusive scan of the counts, one atomic for the tile
    int carry = 0;
    for (int b = 0; b < ntok; b += WAVE) {
      const int c = b + tid < ntok ? t_cnt[b + tid] : 0;
      int x = c;
#pragma unroll
      for (int d = 1; d < WAVE; d <<= 1) {
        const int y = __shfl_up(x, d, WAVE);
        if (tid >= d) x += y;
      }
      if (b + tid < ntok) t_off[b + tid] = carry + x - c;
      carry += __shfl(x, WAVE - 1, WAVE);
    }
    if (tid == 0) base_s = atomicAdd(&a.stats[ST_CANDS], carry);
  }
  __syncthreads();
  const int gw = (tid & (WAVE - 1)) / GG;  // the group's place in its wavefront
  for (int t0 = 0; t0 < ntok; t0 += GTOK) {
    const int g = g0 + t0 + grp;
    const bool valid = g < a.T;
    const int gs = valid ? g : 0;
    const float xn = a.xn[gs];
    const float tau = t_tau[t0 + grp];
    const int tb = base_s + t_off[t0 + grp];
    if (valid && gl == 0) {
      a.tok_base[g] = tb;
      a.tok_n[g] = t_cnt[t0 + grp];
    }
    int run = 0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = gl + GG * i;
      bool c = false;
      if (valid && e < a.E) {
        float l, d;
        interval(a, gs, e, xn, l, d);
        c = l + d >= tau;
      }
      const uint32_t gm = (uint32_t)(__ballot(c) >> (gw * GG)) & ((1u << GG) - 1);
      if (c) {
        const int pos = tb + run + __builtin_popcount(gm & ((1u << gl) - 1));
        a.ch_g[pos] = g;
        a.ch_e[pos] = e;
      }
      run += __builtin_popcount(gm);
    }
  }
}

// Approximate logits of 32 tokens, then their candidates: the workgroup's
// logits and norms are in memory after the barrier (workgroup scope), so the
// candidate pass needs no launch of its own.
// E <= 32 with a multiple of 64 values of H per wavefront: the same sums,
// with x and the gate rows staged through a per-wavefront LDS ring by direct
// global->LDS loads in which 8 lanes fetch one row's 128 contiguous bytes
// (a load instruction covers 8 rows instead of 32 scattered pieces).  Rows
// are 64 values (128 bytes) per stage, their 16-byte granules XOR-swizzled
// by the row index; lane l reads granule 2t + (l >> 5) of row l & 31 for the
// t-th 16-deep MFMA step of a stage.  Token rows past T and gate rows past E
// repeat the last valid row; their sums are not stored.
constexpr int GS_ST = 3;                  // ring stages per wavefront
constexpr int GS_OPB = 32 * 128;          // bytes per operand and stage
constexpr int GS_SB = 2 * GS_OPB;         // bytes per stage
__device__ __forceinline__ void gate_mfma_staged(const GateArgs& a, char* ring_all, float (*red)[32 * 32 * 4],
                                                 float (*ssr)[64]) {
  const int lane = gemm::lane_here(), wave = gemm::opaque((int)(threadIdx.x / WAVE));
  const int g0 = blockIdx.x * 32;
  const int hq = a.H / GATE_WAVES;  // a multiple of 64 here
  const int hbeg = wave * hq;
  const int nb = hq / 64;
  char* ring = ring_all + wave * (GS_ST * GS_SB);
  const uint32_t ring0 = gemm::lds_u32(ring);
  uint32_t xo[4], wo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = i * 8 + (lane >> 3);
    const int gr = (lane & 7) ^ (r & 7);
    const int g = min(g0 + r, a.T - 1), e = min(r, a.E - 1);
    xo[i] = ((uint32_t)g * (uint32_t)a.H + (uint32_t)hbeg) * 2u + (uint32_t)(gr * 16);
    wo[i] = ((uint32_t)e * (uint32_t)a.H + (uint32_t)hbeg) * 2u + (uint32_t)(gr * 16);
  }
  const char* xb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.x));
  const char* wb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.wgt));
  auto issue = [&](int b) {
    const uint32_t st = ring0 + (uint32_t)((b % GS_ST) * GS_SB);
#pragma unroll
    for (int i = 0; i < 4; ++i) gemm::dma16(xb + (size_t)b * 128, xo[i], st + i * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) gemm::dma16(wb + (size_t)b * 128, wo[i], st + GS_OPB + i * 1024);
  };
  for (int b = 0; b < GS_ST - 1 && b < nb; ++b) issue(b);
  f32x16_t acc = f32x16_t{};
  float ss = 0.0f;
  const int row = lane & 31, half = lane >> 5;
  for (int b = 0; b < nb; ++b) {
    const int later = min(nb - 1 - b, GS_ST - 2);
    if (later >= 2) gemm::wait_vm<16>();
    else if (later == 1) gemm::wait_vm<8>();
    else gemm::wait_vm<0>();
    const char* st = ring + (b % GS_ST) * GS_SB + row * 128;
    bf16x8_t xa[4], wa[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int slot = (2 * t + half) ^ (row & 7);
      xa[t] = *reinterpret_cast<const bf16x8_t*>(st + slot * 16);
      wa[t] = *reinterpret_cast<const bf16x8_t*>(st + GS_OPB + slot * 16);
    }
    // the reads of the stage about to be refilled (read one step ago) are done
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    if (b + GS_ST - 1 < nb) issue(b + GS_ST - 1);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float f = (float)xa[t][q];
        ss += f * f;
      }
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[t], wa[t], acc, 0, 0, 0);
    }
  }
  // add the quarters: C[8 (r >> 2) + 4 (l >> 5) + (r & 3)][l & 31]
  if (wave > 0) {
#pragma unroll
    for (int r = 0; r < 16; ++r) red[wave - 1][r * WAVE + lane] = acc[r];
  }
  ssr[wave][lane] = ss;
  __syncthreads();
  if (wave == 0) {
    const int e = lane & 31;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float v = acc[r];
#pragma unroll
      for (int w = 0; w < GATE_WAVES - 1; ++w) v += red[w][r * WAVE + lane];
      const int gr = g0 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (e < a.E && gr < a.T) a.lt[(size_t)gr * a.E + e] = v;
    }
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < GATE_WAVES; ++w) t += ssr[w][lane] + ssr[w][lane ^ 32];
    if (lane < 32 && g0 + lane < a.T) a.xn[g0 + lane] = sqrtf(t);
  }
}

__global__ void __launch_bounds__(GATE_WAVES * WAVE) gate_mfma_kernel(GateArgs a) {
  static_assert(GATE_WAVES * WAVE == NTH && 32 % GTOK == 0, "candidate pass geometry");
  __shared__ int t_cnt[32], t_off[32];
  __shared__ float t_tau[32];
  __shared__ int base_s;
  __shared__ float red[GATE_WAVES - 1][32 * 32 * 4];
  __shared__ float ssr[GATE_WAVES][64];
  __shared__ __align__(16) char ring[GATE_WAVES * GS_ST * GS_SB];
  // E <= 32 (more experts: gate_tile_kernel)
  if ((a.H / GATE_WAVES) % 64 == 0) gate_mfma_staged(a, ring, red, ssr);
  else gate_mfma_body<1, 8, GATE_WAVES>(a, red, ssr);
  __syncthreads();
  cand_tile<2>(a, blockIdx.x * 32, 32, t_cnt, t_off, t_tau, base_s);  // E <= 32: two experts per lane
}

// E > 32: the approximate logits of a tile of GT_M tokens x GT_N experts per
// pass over the experts, on v_mfma_f32_32x32x16_bf16 (fp32 accumulation) with
// both operands streamed through an LDS ring of GT_NS stages of 64-deep
// k-steps by direct global->LDS loads.  In a load instruction 8 lanes fetch
// one row's 128 contiguous bytes, so it covers 8 whole lines (x is row-major
// with 2H-byte rows, the transposed gate too).  A row's 16-byte granules are
// stored XOR-swizzled by (row & 7), so that the fragment reads of 8 lanes on
// 8 consecutive rows hit distinct banks.  Four wavefronts in a 2 x 2 grid,
// each (GT_M / 2) tokens x 64 experts.  Token rows past T and gate rows past
// E repeat the last valid row; their sums are not stored.  The token norms
// come from the same x fragments (wavefronts of the first expert column, on
// the first pass).  Then the candidate pass of the tile's tokens.
constexpr int GT_N = 128;  // experts per pass
constexpr int GT_K = 64;   // values per row piece of a stage (128 bytes)
constexpr int GT_NS = 4;   // ring stages

template <int OUT>
__device__ __forceinline__ void gt_wait(int outstanding) {
  // at most `outstanding` stages (OUT DMA instructions each) still in flight
  if (outstanding >= 2) gemm::wait_vm<2 * OUT>();
  else if (outstanding == 1) gemm::wait_vm<OUT>();
  else gemm::wait_vm<0>();
}

template <int GT_M, int EPL>
__global__ void __launch_bounds__(NTH) gate_tile_kernel(GateArgs a) {
  static_assert(NTH == 4 * WAVE && GT_M % 64 == 0 && GT_M % GTOK == 0, "gate tile geometry");
  constexpr int A_B = GT_M * 2 * GT_K, B_B = GT_N * 2 * GT_K, ST_B = A_B + B_B;
  constexpr int A_I = A_B / 1024 / 4, B_I = B_B / 1024 / 4;  // DMA instructions per wavefront and stage
  constexpr int WI = A_I + B_I;
  constexpr int MBW = GT_M / 64;  // 32-token blocks per wavefront
  static_assert(GT_NS - 2 <= 2, "gt_wait covers two stages in flight");
  __shared__ __attribute__((aligned(1024))) char ring[GT_NS * ST_B];
  __shared__ int t_cnt[GT_M], t_off[GT_M];
  __shared__ float t_tau[GT_M];
  __shared__ int base_s;
  const int lane = gemm::lane_here(), wave = gemm::opaque((int)(threadIdx.x / WAVE));
  const int wm = wave & 1, wn = wave >> 1;
  const int g0 = blockIdx.x * GT_M;
  const int H = gemm::opaque(a.H), nk = H / GT_K;
  const uint32_t ring0 = (uint32_t)gemm::opaque((int)gemm::lds_u32(ring));
  // this lane's byte offsets of its DMA rows from the operands' first rows
  uint32_t ao[A_I];
#pragma unroll
  for (int i = 0; i < A_I; ++i) {
    const int row = (wave * A_I + i) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7);
    ao[i] = (uint32_t)(min(row, a.T - 1 - g0) * H * 2 + c * 16);
  }
  const char* xb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.x + (size_t)g0 * H));
  float ss[MBW];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) ss[mb] = 0.0f;
  for (int eb = 0; eb < a.E; eb += GT_N) {
    uint32_t bo[B_I];
#pragma unroll
    for (int i = 0; i < B_I; ++i) {
      const int row = (wave * B_I + i) * 8 + (lane >> 3);
      const int c = (lane & 7) ^ (row & 7);
      bo[i] = (uint32_t)(min(row, a.E - 1 - eb) * H * 2 + c * 16);
    }
    const char* wb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.wgt + (size_t)eb * H));
    auto issue = [&](int st) {
      const uint32_t dst = ring0 + (uint32_t)((st % GT_NS) * ST_B);
#pragma unroll
      for (int i = 0; i < A_I; ++i) gemm::dma16(xb + (size_t)st * (2 * GT_K), ao[i], dst + (wave * A_I + i) * 1024);
#pragma unroll
      for (int i = 0; i < B_I; ++i)
        gemm::dma16(wb + (size_t)st * (2 * GT_K), bo[i], dst + A_B + (wave * B_I + i) * 1024);
    };
    f32x16_t acc[MBW][2];
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = f32x16_t{};
    for (int st = 0; st < GT_NS - 1 && st < nk; ++st) issue(st);
    const int ra = wm * (GT_M / 2) + (lane & 31), rb = wn * 64 + (lane & 31);
    for (int st = 0; st < nk; ++st) {
      gt_wait<WI>(min(GT_NS - 2, nk - 1 - st));
      __builtin_amdgcn_s_barrier();
      gemm::compiler_fence();
      if (st + GT_NS - 1 < nk) issue(st + GT_NS - 1);
      const char* sa = ring + (st % GT_NS) * ST_B;
      const char* sb = sa + A_B;
#pragma unroll
      for (int kk = 0; kk < GT_K / 16; ++kk) {
        const int ch = 2 * kk + (lane >> 5);
        bf16x8_t af[MBW], bf[2];
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb) {
          const int r = ra + mb * 32;
          af[mb] = *reinterpret_cast<const bf16x8_t*>(sa + r * 128 + ((ch ^ (r & 7)) << 4));
        }
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int r = rb + nb * 32;
          bf[nb] = *reinterpret_cast<const bf16x8_t*>(sb + r * 128 + ((ch ^ (r & 7)) << 4));
        }
        if (wn == 0 && eb == 0) {
#pragma unroll
          for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              const float f = (float)af[mb][q];
              ss[mb] += f * f;
            }
        }
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bf[nb], acc[mb][nb], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_barrier();  // the ring is refilled by the next pass
    gemm::compiler_fence();
    // C[8 (r >> 2) + 4 (l >> 5) + (r & 3)][l & 31] of each 32 x 32 block
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int e = eb + wn * 64 + nb * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int g = g0 + wm * (GT_M / 2) + mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (e < a.E && g < a.T) a.lt[(size_t)g * a.E + e] = acc[mb][nb][r];
        }
      }
  }
  if (wn == 0) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb) {
      const float t = ss[mb] + __shfl_xor(ss[mb], 32, WAVE);
      const int g = g0 + wm * (GT_M / 2) + mb * 32 + lane;
      if (lane < 32 && g < a.T) a.xn[g] = sqrtf(t);
    }
  }
  __syncthreads();  // the tile's logits and norms are in memory for the candidate pass
  cand_tile<EPL>(a, g0, GT_M, t_cnt, t_off, t_tau, base_s);
}

template __global__ void gate_tile_kernel<64, 4>(GateArgs);
template __global__ void gate_tile_kernel<64, 8>(GateArgs);
template __global__ void gate_tile_kernel<64, 32>(GateArgs);
template __global__ void gate_tile_kernel<128, 4>(GateArgs);
template __global__ void gate_tile_kernel<128, 8>(GateArgs);
template __global__ void gate_tile_kernel<128, 32>(GateArgs);

// 32 < E <= 128: the approximate logits of GT_M tokens x all experts in one
// workgroup of 8 wavefronts, then the candidate pass, without the logits
// leaving LDS.  The operands stream through the same LDS ring as in
// gate_tile_kernel (64-deep k-steps, 8 lanes per 128-byte row piece, granules
// XOR-swizzled by row & 7).  Wavefronts 0-3 take the first two 16-deep
// slices of every k-step, 4-7 the last two, in a 2 x 2 grid of (GT_M / 2)
// tokens x 64 experts each; the two halves' sums are added through LDS at
// the end (the bound holds for any order of the approximate sum).  The
// logits, plus bias, go to an LDS tile of GT_M rows (padded to 129 words so
// that lanes reading their own rows hit distinct banks); one lane per token
// then keeps the k largest lower ends of its intervals in a sorted list,
// takes tau = the k-th, and lists the experts whose upper end reaches tau.
constexpr int G2_PAD = GT_N + 1;  // words per row of the LDS logit tile

template <int GT_M>
__global__ void __launch_bounds__(2 * NTH) gate_tile2_kernel(GateArgs a) {
  constexpr int NW = 8;
  constexpr int A_B = GT_M * 2 * GT_K, B_B = GT_N * 2 * GT_K, ST_B = A_B + B_B;
  constexpr int A_I = A_B / 1024 / NW, B_I = B_B / 1024 / NW;  // DMA instructions per wavefront and stage
  constexpr int WI = A_I + B_I;
  constexpr int MBW = GT_M / 64;
  static_assert(A_I >= 1 && B_I >= 1 && GT_M % 64 == 0, "tile geometry");
  static_assert(GT_M * G2_PAD * 4 <= GT_NS * ST_B && 4 * MBW * 2 * 16 * WAVE * 4 <= GT_NS * ST_B, "ring reuse");
  __shared__ __attribute__((aligned(1024))) char ring[GT_NS * ST_B];
  __shared__ float ssq[2][GT_M];  // partial squared norms of the two k halves
  __shared__ float bias_s[GT_N], wn_s[GT_N];
  __shared__ int t_cnt[GT_M], t_off[GT_M];
  __shared__ int base_s;
  const int lane = gemm::lane_here(), wave = gemm::opaque((int)(threadIdx.x / WAVE));
  const int kh = wave >> 2, wm = wave & 1, wn = (wave >> 1) & 1;
  const int g0 = blockIdx.x * GT_M;
  const int H = gemm::opaque(a.H), nk = H / GT_K;
  const uint32_t ring0 = (uint32_t)gemm::opaque((int)gemm::lds_u32(ring));
  for (int e = threadIdx.x; e < GT_N; e += 2 * NTH) {
    bias_s[e] = (a.bias && e < a.E) ? a.bias[e] : 0.0f;
    wn_s[e] = e < a.E ? a.wn[e] : 0.0f;
  }
  uint32_t ao[A_I], bo[B_I];
#pragma unroll
  for (int i = 0; i < A_I; ++i) {
    const int row = (wave * A_I + i) * 8 + (lane >> 3);
    ao[i] = (uint32_t)(min(row, a.T - 1 - g0) * H * 2 + (((lane & 7) ^ (row & 7)) << 4));
  }
#pragma unroll
  for (int i = 0; i < B_I; ++i) {
    const int row = (wave * B_I + i) * 8 + (lane >> 3);
    bo[i] = (uint32_t)(min(row, a.E - 1) * H * 2 + (((lane & 7) ^ (row & 7)) << 4));
  }
  const char* xb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.x + (size_t)g0 * H));
  const char* wb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.wgt));
  auto issue = [&](int st) {
    const uint32_t dst = ring0 + (uint32_t)((st % GT_NS) * ST_B);
#pragma unroll
    for (int i = 0; i < A_I; ++i) gemm::dma16(xb + (size_t)st * (2 * GT_K), ao[i], dst + (wave * A_I + i) * 1024);
#pragma unroll
    for (int i = 0; i < B_I; ++i)
      gemm::dma16(wb + (size_t)st * (2 * GT_K), bo[i], dst + A_B + (wave * B_I + i) * 1024);
  };
  f32x16_t acc[MBW][2];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = f32x16_t{};
  float ss[MBW];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) ss[mb] = 0.0f;
  for (int st = 0; st < GT_NS - 1 && st < nk; ++st) issue(st);
  const int ra = wm * (GT_M / 2) + (lane & 31), rb = wn * 64 + (lane & 31);
  for (int st = 0; st < nk; ++st) {
    gt_wait<WI>(min(GT_NS - 2, nk - 1 - st));
    __builtin_amdgcn_s_barrier();
    gemm::compiler_fence();
    if (st + GT_NS - 1 < nk) issue(st + GT_NS - 1);
    const char* sa = ring + (st % GT_NS) * ST_B;
    const char* sb = sa + A_B;
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int ch = 2 * (2 * kh + k2) + (lane >> 5);
      bf16x8_t af[MBW], bf[2];
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb) {
        const int r = ra + mb * 32;
        af[mb] = *reinterpret_cast<const bf16x8_t*>(sa + r * 128 + ((ch ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int r = rb + nb * 32;
        bf[nb] = *reinterpret_cast<const bf16x8_t*>(sb + r * 128 + ((ch ^ (r & 7)) << 4));
      }
      if (wn == 0) {
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float f = (float)af[mb][q];
            ss[mb] += f * f;
          }
      }
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bf[nb], acc[mb][nb], 0, 0, 0);
    }
  }
  __builtin_amdgcn_s_barrier();  // the ring is reused below
  gemm::compiler_fence();
  // the second k half's sums, through LDS, into the first half's
  float* part = reinterpret_cast<float*>(ring);
  const int pw = wave & 3;  // the partner wavefront's place in its half
  if (kh == 1) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) part[(((pw * MBW + mb) * 2 + nb) * 16 + r) * WAVE + lane] = acc[mb][nb][r];
  }
  if (wn == 0) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb) {
      const float t = ss[mb] + __shfl_xor(ss[mb], 32, WAVE);
      if (lane < 32) ssq[kh][wm * (GT_M / 2) + mb * 32 + lane] = t;
    }
  }
  __syncthreads();
  if (kh == 0) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mb][nb][r] += part[(((pw * MBW + mb) * 2 + nb) * 16 + r) * WAVE + lane];
  }
  __syncthreads();
  // logits plus bias into the tile: C[8 (r >> 2) + 4 (l >> 5) + (r & 3)][l & 31] of each block
  float* tile = reinterpret_cast<float*>(ring);
  if (kh == 0) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int e = wn * 64 + nb * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int t = wm * (GT_M / 2) + mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          float l = acc[mb][nb][r];
          if (a.bias) l = l + bias_s[e];
          tile[t * G2_PAD + e] = l;
        }
      }
  }
  __syncthreads();
  // candidates, LPT adjacent lanes per token (lane q takes experts
  // [q * EQ, q * EQ + EQ)): each keeps the k largest lower ends of its
  // experts in a sorted list (equal values all kept) and the upper ends in
  // registers; the lists are merged across the token's lanes, so top[k-1] is
  // the k-th largest lower end over every expert; then the experts whose
  // upper end reaches it, in expert order
  constexpr int LPT = 2 * NTH / GT_M, EQ = GT_N / LPT;
  static_assert(LPT * GT_M == 2 * NTH && (LPT & (LPT - 1)) == 0 && LPT <= WAVE, "lanes per token");
  const int tq = threadIdx.x / LPT, q = threadIdx.x % LPT;
  const int g = g0 + tq;
  const bool mine = g < a.T;
  float top[MAX_TOPK];
#pragma unroll
  for (int j = 0; j < MAX_TOPK; ++j) top[j] = -INFINITY;
  auto insert = [&](float v) {
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j) {
      const float hi = fmaxf(v, top[j]);
      v = fminf(v, top[j]);
      top[j] = hi;
    }
  };
  float up[EQ];
  if (mine) {
    const float xn = sqrtf(ssq[0][tq] + ssq[1][tq]);
#pragma unroll
    for (int i = 0; i < EQ; ++i) {
      const int e = q * EQ + i;
      up[i] = -INFINITY;
      if (e < a.E) {
        const float l = tile[tq * G2_PAD + e];
        float d = a.bound * xn * wn_s[e];
        d = d + 4.0f * 5.9604645e-8f * (fabsf(l) + d) + 1e-30f;
        insert(l - d);
        up[i] = l + d;
      }
    }
  }
#pragma unroll
  for (int m = 1; m < LPT; m <<= 1) {
    float other[MAX_TOPK];
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j) other[j] = __shfl_xor(top[j], m, WAVE);
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j) insert(other[j]);
  }
  float tau = -INFINITY;
#pragma unroll
  for (int j = 0; j < MAX_TOPK; ++j)
    if (j == a.k - 1) tau = top[j];
  int cnt = 0;
  if (mine) {
#pragma unroll
    for (int i = 0; i < EQ; ++i) cnt += (q * EQ + i < a.E && up[i] >= tau) ? 1 : 0;
  }
  // this lane's place among its token's candidates, and the token's count
  int incl = cnt;
#pragma unroll
  for (int m = 1; m < LPT; m <<= 1) {
    const int y = __shfl_up(incl, m, WAVE);
    if (q >= m) incl += y;
  }
  const int ntok = __shfl(incl, (lane | (LPT - 1)), WAVE);
  if (q == 0) t_cnt[tq] = ntok;  // 0 for rows past T
  __syncthreads();
  if (threadIdx.x < WAVE) {  // exclusive scan of the counts, one atomic for the tile
    int carry = 0;
    for (int b = 0; b < GT_M; b += WAVE) {
      const int c = t_cnt[b + lane];
      int x = c;
#pragma unroll
      for (int d = 1; d < WAVE; d <<= 1) {
        const int y = __shfl_up(x, d, WAVE);
        if (lane >= d) x += y;
      }
      t_off[b + lane] = carry + x - c;
      carry += __shfl(x, WAVE - 1, WAVE);
    }
    if (lane == 0) base_s = atomicAdd(&a.stats[ST_CANDS], carry);
  }
  __syncthreads();
  if (mine) {
    const int tb = base_s + t_off[tq];
    if (q == 0) {
      a.tok_base[g] = tb;
      a.tok_n[g] = ntok;
    }
    int pos = tb + incl - cnt;
#pragma unroll
    for (int i = 0; i < EQ; ++i) {
      const int e = q * EQ + i;
      if (e < a.E && up[i] >= tau) {
        a.ch_g[pos] = g;
        a.ch_e[pos] = e;
        ++pos;
      }
    }
  }
}

template __global__ void gate_tile2_kernel<64>(GateArgs);
template __global__ void gate_tile2_kernel<128>(GateArgs);

// the defined logit of one (token, expert): fp32, one accumulator, h
// ascending, each product rounded before the add.  A product of two bf16
// values is exact in fp32, so fma(x, w, acc) rounds exactly as acc + x*w and
// saves the multiply on the serial chain.  Two register sets of PF vectors
// take turns so that the next block's loads are in flight while the current
// one is added.
constexpr int PF = 16;
__device__ __forceinline__ void chain_add(float& acc, const u32x4_t (&xb)[PF], const u32x4_t (&wb)[PF]) {
#pragma unroll
  for (int i = 0; i < PF; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc = __builtin_fmaf(bf16_lo(xb[i][q]), bf16_lo(wb[i][q]), acc);
      acc = __builtin_fmaf(bf16_hi(xb[i][q]), bf16_hi(wb[i][q]), acc);
    }
}
__device__ __forceinline__ float exact_logit(const uint16_t* xr, const uint16_t* wr, int H) {
  const u32x4_t* xv = reinterpret_cast<const u32x4_t*>(xr);
  const u32x4_t* wv = reinterpret_cast<const u32x4_t*>(wr);
  const int nv = H >> 3;       // 16-byte vectors per row
  const int nb = nv / PF;      // whole blocks of PF vectors
  u32x4_t xa[PF], wa[PF], xb[PF], wb[PF];
  auto load = [&](u32x4_t (&xd)[PF], u32x4_t (&wd)[PF], int blk) {
#pragma unroll
    for (int i = 0; i < PF; ++i) { xd[i] = xv[blk * PF + i]; wd[i] = wv[blk * PF + i]; }
  };
  float acc = 0.0f;
  if (nb > 0) load(xa, wa, 0);
  for (int b = 0; b < nb; b += 2) {
    if (b + 1 < nb) load(xb, wb, b + 1);
    chain_add(acc, xa, wa);
    if (b + 1 < nb) {
      if (b + 2 < nb) load(xa, wa, b + 2);
      chain_add(acc, xb, wb);
    }
  }
  for (int v = nb * PF; v < nv; ++v) {  // the vectors after the last whole block
    const u32x4_t x = xv[v], w = wv[v];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc = __builtin_fmaf(bf16_lo(x[q]), bf16_lo(w[q]), acc);
      acc = __builtin_fmaf(bf16_hi(x[q]), bf16_hi(w[q]), acc);
    }
  }
  return acc;
}

// one lane per chain of the list, one wavefront per workgroup: each chain
// streams two rows of H bf16 values, so the chains are spread over as many
// CUs as possible (a CU's memory pipeline, not its VALU, bounds a chain)
__global__ void __launch_bounds__(WAVE) gate_chain_kernel(GateArgs a) {
  const int n = a.stats[ST_CANDS];
  for (int i = blockIdx.x * WAVE + threadIdx.x; i < n; i += gridDim.x * WAVE) {
    const int g = a.ch_g[i], e = a.ch_e[i];
    float l = exact_logit(a.x + (size_t)g * a.H, a.wgt + (size_t)e * a.H, a.H);
    if (a.bias) l = l + a.bias[e];
    a.ch_l[i] = l;
  }
}

// The chains of the list for E <= CH_E: one lane per chain, CH_W chains per
// workgroup.  The chains of one token are adjacent in the list and every
// token has at least k of them (its top k are among them), so a range of
// CH_W chains holds at most CH_W / k + 2 tokens, CX of them in a stage.  For
// each 64-value block of h the workgroup stages in LDS that block of all gate
// rows (CH_E rows of 128 bytes, rows past E repeating the last one) and of the
// x rows of its tokens (CX rows, slots past the range's tokens repeating its
// first), whole lines by direct global->LDS loads, in a ring of NP stages: no
// operand goes through registers ahead of its use, so with NP = 3 two blocks
// are in flight while one is added, and two workgroups share a CU.  A lane
// reads its token's x and its expert's gate values from the stage and adds
// the 64 products in order, one fused multiply-add each: the product of two
// bf16 values is exact in fp32, so this is the product rounded, then the sum
// rounded, as in exact_logit.  Granules of a staged row are XOR-swizzled
// (chain_swz).
constexpr int CH_W = 512, CH_E = 128, CH_K = 64;
constexpr int CH_NW = CH_W / WAVE;       // wavefronts per workgroup
constexpr int CH_WB = CH_E * 2 * CH_K;   // gate bytes of a stage
constexpr int CH_DMA = CH_E / 8 / CH_NW; // gate DMA instructions per wavefront and block

// Granule swizzle of a staged 128-byte row: two rows share a 256-byte bank
// window, so the granule is XOR-ed with bits 1-3 of the row, and rows that
// differ in their low four bits put a given granule in different banks.
__device__ __forceinline__ int chain_swz(int row) { return (row >> 1) & 7; }

template <int CX, int NP>
struct ChainGeo {
  static constexpr int STAGE = CH_WB + CX * 2 * CH_K;        // bytes of a stage
  static constexpr int XI = (CX / 8 + CH_NW - 1) / CH_NW;    // x DMA instructions per wavefront and block (at most)
  static_assert(CX % 8 == 0 && STAGE % 1024 == 0 && (NP == 2 || NP == 3), "chain staging geometry");
};

// One range of CH_W chains from c0 (< n); the range's chains belong to at
// most CX tokens (the host picks CX from k).
template <int CX, int NP>
__device__ __forceinline__ void chain_range(const GateArgs& a, char* ring, int* tok, int* wsum, int c0, int n) {
  using Geo = ChainGeo<CX, NP>;
  const int lane = gemm::lane_here(), wave = gemm::opaque((int)(threadIdx.x / WAVE));
  const int i = c0 + (int)threadIdx.x;
  const bool live = i < n;
  const int ic = live ? i : n - 1;
  const int g = a.ch_g[ic], e = a.ch_e[ic];
  // the range's tokens, in list order: a live lane starts a slot where its
  // token differs from the previous entry's (the range's first entry always)
  const bool head = live && (i == c0 || a.ch_g[i - 1] != g);
  const uint64_t hm = __builtin_amdgcn_ballot_w64(head);
  const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(hm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)hm, 0));
  if (lane == 0) wsum[wave] = __builtin_popcountll(hm);
  __syncthreads();
  int base = 0, nslot = 0;
  for (int w = 0; w < CH_NW; ++w) {
    const int c = wsum[w];
    if (w < wave) base += c;
    nslot += c;
  }
  if (nslot > CX) {
    // more tokens than a stage holds (not expected: every token has at least
    // k chains): each lane evaluates its chain straight from global memory
    if (live) {
      const u32x4_t* xv = reinterpret_cast<const u32x4_t*>(a.x + (size_t)g * a.H);
      const u32x4_t* wv = reinterpret_cast<const u32x4_t*>(a.wgt + (size_t)e * a.H);
      float l = 0.0f;
      for (int v = 0; v < (a.H >> 3); ++v) {
        const u32x4_t xq = xv[v], wq = wv[v];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          l = __builtin_fmaf(bf16_lo(xq[q]), bf16_lo(wq[q]), l);
          l = __builtin_fmaf(bf16_hi(xq[q]), bf16_hi(wq[q]), l);
        }
      }
      a.ch_l[i] = a.bias ? l + a.bias[e] : l;
    }
    __syncthreads();
    return;
  }
  const int slot = base + before - (head ? 0 : 1);
  if (head) tok[slot] = g;
  __syncthreads();
  const int H = gemm::opaque(a.H), nb = H / CH_K;
  const uint32_t ring0 = (uint32_t)gemm::opaque((int)gemm::lds_u32(ring));
  uint32_t wo[CH_DMA], xo[Geo::XI];
#pragma unroll
  for (int j = 0; j < CH_DMA; ++j) {
    const int row = (wave * CH_DMA + j) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ chain_swz(row);
    wo[j] = (uint32_t)(min(row, a.E - 1) * H * 2 + c * 16);
  }
#pragma unroll
  for (int j = 0; j < Geo::XI; ++j) {
    const int row = (j * CH_NW + wave) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ chain_swz(row);
    xo[j] = (uint32_t)(tok[row < nslot ? row : 0] * H * 2 + c * 16);
  }
  // x DMA instructions of this wavefront: Geo::XI, or one fewer where the
  // last round of 8-row instructions does not reach it
  const int nxi = gemm::opaque((CX / 8 - wave + CH_NW - 1) / CH_NW);
  const char* wb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.wgt));
  const char* xb = gemm::uniform_ptr(reinterpret_cast<const char*>(a.x));
  auto issue = [&](int b) {
    const uint32_t st = ring0 + (uint32_t)((b % NP) * Geo::STAGE);
#pragma unroll
    for (int j = 0; j < CH_DMA; ++j) gemm::dma16(wb + (size_t)b * (2 * CH_K), wo[j], st + (wave * CH_DMA + j) * 1024);
#pragma unroll
    for (int j = 0; j < Geo::XI; ++j)
      if (j < nxi) gemm::dma16(xb + (size_t)b * (2 * CH_K), xo[j], st + CH_WB + (j * CH_NW + wave) * 1024);
  };
  float acc = 0.0f;
  // this lane's 16 granule offsets within a stage (its x row and its gate
  // row, swizzled), computed once: with the stage index a constant (the
  // block loop below runs NP blocks per iteration) every read is one of
  // these plus an immediate
  int xg[8], wg[8];
  {
    const int wrow = e * (2 * CH_K), wsw = chain_swz(e);
    const int xrow = CH_WB + slot * (2 * CH_K), xsw = chain_swz(slot);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      xg[q] = xrow + ((q ^ xsw) << 4);
      wg[q] = wrow + ((q ^ wsw) << 4);
    }
  }
  // block b, in stage sb = b mod NP: the stage holds this wavefront's loads
  // once at most the blocks issued after it are outstanding; past the
  // barrier every wavefront's have landed and every wavefront has added
  // block b - 1, so the stage of block b + NP - 1 (that of b - 1) is
  // refilled, then block b is added
  auto step = [&](int b, int sb) {
    if (NP == 3 && b + 1 < nb) {
      if (nxi == Geo::XI) gemm::wait_vm<CH_DMA + Geo::XI>(); else gemm::wait_vm<CH_DMA + Geo::XI - 1>();
    } else {
      gemm::wait_vm<0>();
    }
    __builtin_amdgcn_s_barrier();
    gemm::compiler_fence();
    if (b + NP - 1 < nb) issue(b + NP - 1);
    const char* st = ring + sb * Geo::STAGE;
    u32x4_t xv[8], wv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      xv[q] = *reinterpret_cast<const u32x4_t*>(st + xg[q]);
      wv[q] = *reinterpret_cast<const u32x4_t*>(st + wg[q]);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        acc = __builtin_fmaf(bf16_lo(xv[q][r]), bf16_lo(wv[q][r]), acc);
        acc = __builtin_fmaf(bf16_hi(xv[q][r]), bf16_hi(wv[q][r]), acc);
      }
    // the block's adds complete here, before the next block's barrier (the
    // compiler would otherwise interleave them with the next block's reads
    // and hold both blocks' operands at once)
    asm volatile("" : "+v"(acc));
  };
  for (int b = 0; b < NP - 1 && b < nb; ++b) issue(b);
  int b = 0;
  for (; b + NP <= nb; b += NP) {
#pragma unroll
    for (int sb = 0; sb < NP; ++sb) step(b + sb, sb);
  }
  for (int sb = 0; b < nb; ++b, ++sb) step(b, sb);
  if (live) a.ch_l[i] = a.bias ? acc + a.bias[e] : acc;
  // the next range refills every stage and rewrites the slot table
  __syncthreads();
}

// Persistent over the ranges of CH_W chains (the chain count is known only
// on the device).  Two workgroups per CU: 4 wavefronts per SIMD.
template <int CX, int NP>
__global__ void __launch_bounds__(CH_W, 4) gate_chain_staged_kernel(GateArgs a) {
  static_assert(CH_E % (8 * CH_NW) == 0, "gate rows per DMA round");
  __shared__ __attribute__((aligned(1024))) char ring[NP * ChainGeo<CX, NP>::STAGE];
  __shared__ int tok[CX];
  __shared__ int wsum[CH_NW];
  const int n = a.stats[ST_CANDS];
  for (int c0 = blockIdx.x * CH_W; c0 < n; c0 += gridDim.x * CH_W) chain_range<CX, NP>(a, ring, tok, wsum, c0, n);
}

template __global__ void gate_chain_staged_kernel<72, 3>(GateArgs);
template __global__ void gate_chain_staged_kernel<136, 2>(GateArgs);

// Counts the local selections of this block's tokens per local expert into
// blk_cnt (one table block = NTH tokens) and the tokens with an invalid or
// repeated id into blk_bad; ids: this thread's token's k ids (valid: g < T).
__device__ __forceinline__ void count_block(const TableArgs& t, const int* ids, bool valid);

// top-k of the candidates' defined logits (descending, equal logits ->
// smaller id), one lane per token keeping a sorted list of the k best, then
// the renormalised softmax weights of the chosen experts: exp(l_j - m) over
// their sum (the normaliser over all experts cancels in the renormalisation,
// so it is not formed).  COUNT: the routing tables' first step on the ids
// just chosen (the table blocks are these workgroups' tokens), as
// tab_count_kernel would do it on topk_idx.
template <int EPL, bool COUNT>
__global__ void __launch_bounds__(NTH) gate_final_kernel(GateArgs a, TableArgs tab) {
  const int g = blockIdx.x * NTH + threadIdx.x;
  const bool valid = g < a.T;
  float tv[MAX_TOPK];
  int ti[MAX_TOPK];
#pragma unroll
  for (int j = 0; j < MAX_TOPK; ++j) { tv[j] = -INFINITY; ti[j] = 1 << 30; }
  if (valid) {
    const int tb = a.tok_base[g], tn = a.tok_n[g];
    // the candidates in batches of CB, every load of a batch in flight
    // before the first insertion (list order, as one at a time)
    constexpr int CB = 16;
    for (int c0 = 0; c0 < tn; c0 += CB) {
      float cv[CB];
      int ce[CB];
#pragma unroll
      for (int i = 0; i < CB; ++i)
        if (c0 + i < tn) {
          cv[i] = a.ch_l[tb + c0 + i];
          ce[i] = a.ch_e[tb + c0 + i];
        }
      for (int i = 0; i < CB; ++i) {
        if (c0 + i >= tn) break;
        float v = cv[i];
        int e = ce[i];
#pragma unroll
        for (int j = 0; j < MAX_TOPK; ++j) {
          if (better(v, e, tv[j], ti[j])) {
            const float ov = tv[j];
            const int oe = ti[j];
            tv[j] = v;
            ti[j] = e;
            v = ov;
            e = oe;
          }
        }
      }
    }
    const float m = tv[0];
    float p[MAX_TOPK];
    float ps = 0.0f;
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j)
      if (j < a.k) { p[j] = expf(tv[j] - m); ps += p[j]; }
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j)
      if (j < a.k) {
        a.topk_idx[(size_t)g * a.k + j] = ti[j];
        a.topk_w[(size_t)g * a.k + j] = p[j] / ps;
      }
  }
  if constexpr (COUNT) count_block(tab, ti, valid);
}

#define MOE_GATE_FINAL(EPL)                                                  \
  template __global__ void gate_final_kernel<EPL, false>(GateArgs, TableArgs); \
  template __global__ void gate_final_kernel<EPL, true>(GateArgs, TableArgs);
MOE_GATE_FINAL(1)
MOE_GATE_FINAL(2)
MOE_GATE_FINAL(4)
MOE_GATE_FINAL(8)
MOE_GATE_FINAL(32)
#undef MOE_GATE_FINAL

// ---------------------------------------------------------------------------
// Routing tables.  A pair (g, j) is local when id = topk_idx[g,j] is in
// [0, E), not repeated earlier in row g, and le = id - e0 is in [0, E_l).
// ---------------------------------------------------------------------------
constexpr int TB = NTH;  // tokens per table block

__device__ inline int local_expert(const TableArgs& a, const int* ids, int j, bool* bad) {
  int id = ids[j];
  if (id < 0 || id >= a.E) { *bad = true; return -1; }
  for (int jj = 0; jj < j; ++jj)
    if (ids[jj] == id) { *bad = true; return -1; }
  int le = id - a.e0;
  return (le >= 0 && le < a.El) ? le : -1;
}

__device__ __forceinline__ void count_block(const TableArgs& a, const int* ids, bool valid) {
  __shared__ int hist[MAX_SEG];
  __shared__ int nbad;
  const int tid = threadIdx.x;
  for (int i = tid; i < a.El; i += NTH) hist[i] = 0;
  if (tid == 0) nbad = 0;
  __syncthreads();
  bool bad = false;
  if (valid) {
    for (int j = 0; j < a.k; ++j) {
      int le = local_expert(a, ids, j, &bad);
      if (le >= 0) atomicAdd(&hist[le], 1);
    }
  }
  if (bad) {
    atomicAdd(&nbad, 1);
    atomicOr(a.err, ERR_ROUTING);
  }
  __syncthreads();
  for (int i = tid; i < a.El; i += NTH) a.blk_cnt[(size_t)blockIdx.x * a.El + i] = hist[i];
  if (tid == 0) a.blk_bad[blockIdx.x] = nbad;
}

__global__ void __launch_bounds__(NTH) tab_count_kernel(TableArgs a) {
  const int g = blockIdx.x * TB + threadIdx.x;
  const bool valid = g < a.T;
  int ids[MAX_TOPK];
  if (valid)
    for (int j = 0; j < a.k; ++j) ids[j] = a.topk_idx[(size_t)g * a.k + j];
  count_block(a, ids, valid);
}

// Expert offsets and each table block's offset within every expert: one
// wavefront per expert scans the block counts 64 at a time.  Also clears
// the unique-token counts (tab_perm adds to them) and writes the chunk
// offsets that need no search (chunk 0 starts at the expert's first slot,
// chunk K ends at its last).
__global__ void __launch_bounds__(TAB_SCAN_THREADS) tab_scan_kernel(TableArgs a) {
  constexpr int NW = TAB_SCAN_THREADS / WAVE;
  __shared__ int tot[MAX_SEG];
  __shared__ int badw[NW];
  __shared__ int offs[MAX_SEG + 1];
  const int tid = threadIdx.x, lane = tid & (WAVE - 1), wave = tid / WAVE;
  for (int le = wave; le < a.El; le += NW) {
    int carry = 0;
    for (int b0 = 0; b0 < a.nblk; b0 += WAVE) {
      const int b = b0 + lane;
      const int c = b < a.nblk ? a.blk_cnt[(size_t)b * a.El + le] : 0;
      int x = c;
#pragma unroll
      for (int d = 1; d < WAVE; d <<= 1) {
        const int y = __shfl_up(x, d, WAVE);
        if (lane >= d) x += y;
      }
      if (b < a.nblk) a.blk_off[(size_t)b * a.El + le] = carry + x - c;
      carry += __shfl(x, WAVE - 1, WAVE);
    }
    if (lane == 0) tot[le] = carry;
  }
  int bad = 0;
  for (int b = tid; b < a.nblk; b += TAB_SCAN_THREADS) bad += a.blk_bad[b];
#pragma unroll
  for (int d = WAVE / 2; d > 0; d >>= 1) bad += __shfl_xor(bad, d, WAVE);
  if (lane == 0) badw[wave] = bad;
  for (int r = tid; r < a.R; r += TAB_SCAN_THREADS) a.uniq[r] = 0;
  __syncthreads();
  if (tid == 0) {
    int s = 0;
    for (int le = 0; le < a.El; ++le) { offs[le] = s; a.off[le] = s; s += tot[le]; }
    offs[a.El] = s;
    a.off[a.El] = s;
    // the table builder's stats words: the bad-id count here, the rest in
    // tab_finalize (words it does not write stay zero)
    int nb = 0;
    for (int w = 0; w < NW; ++w) nb += badw[w];
    for (int w = 0; w < ST_CANDS; ++w) a.stats[w] = w == ST_BADIDS ? nb : 0;
  }
  __syncthreads();
  for (int v = tid; v < KOPT * a.El * SUBW; v += TAB_SCAN_THREADS) {
    const int ki = v / (a.El * SUBW), le = (v / SUBW) % a.El, q = v % SUBW, K = kopt_value(ki);
    // an inner boundary ceil(q T / K) at T (fewer tokens than chunks) is in
    // no table block: every slot of the expert lies before it
    if (q == 0) a.sub_off[v] = offs[le];
    else if (q == K || (q < K && ((long long)q * a.T + K - 1) / K >= a.T)) a.sub_off[v] = offs[le + 1];
    else if (q > K) a.sub_off[v] = 0;
  }
  for (int v = tid; v < a.El; v += TAB_SCAN_THREADS) {
    a.rbnd[v * (a.R + 1)] = offs[v];
    a.rbnd[v * (a.R + 1) + a.R] = offs[v + 1];
  }
}

// Slots, inverse and first slots by wavefront ballots (ranks within a
// block, ordered by token), unique tokens per rank, and the first slot of
// every expert at or after each rank boundary and each inner chunk boundary
// that falls in this block: the expert's offset, plus the block's offset in
// it, plus its selections in the block before the boundary token.
__global__ void __launch_bounds__(NTH) tab_perm_kernel(TableArgs a) {
  constexpr int NW = NTH / WAVE;
  __shared__ int wc[NW][MAX_SEG];
  __shared__ uint64_t mk[NW][MAX_SEG];
  __shared__ int uq[64];
  const int tid = threadIdx.x;
  const int lane = tid & (WAVE - 1);
  const int wave = tid / WAVE;
  const int g = blockIdx.x * TB + tid;
  const bool valid = g < a.T;
  for (int r = tid; r < a.R; r += NTH) uq[r] = 0;

  int le_j[MAX_TOPK], r_j[MAX_TOPK];
  int ids[MAX_TOPK];
  bool bad = false;
#pragma unroll
  for (int j = 0; j < MAX_TOPK; ++j) { le_j[j] = -1; r_j[j] = 0; }
  if (valid) {
    for (int j = 0; j < a.k; ++j) ids[j] = a.topk_idx[(size_t)g * a.k + j];
    for (int j = 0; j < a.k; ++j) le_j[j] = local_expert(a, ids, j, &bad);
  }
  const uint64_t lt_mask = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int le = 0; le < a.El; ++le) {
    bool sel = false;
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j) sel |= (le_j[j] == le);
    uint64_t m = __ballot(sel);
    int rank = __popcll(m & lt_mask);
    if (sel) {
#pragma unroll
      for (int j = 0; j < MAX_TOPK; ++j)
        if (le_j[j] == le) r_j[j] = rank;
    }
    if (lane == 0) {
      wc[wave][le] = __popcll(m);
      mk[wave][le] = m;
    }
  }
  __syncthreads();
  // boundaries: rank r*Tr (0 < r < R), then the inner chunk boundaries
  // ceil(q*T/K) (0 < q < K) of K = 2, 4, 8; chunk(g) = floor(g*K/T) >= q
  // exactly when g >= ceil(q*T/K)
  {
    const int t0 = blockIdx.x * TB, t1 = min(a.T, t0 + TB);
    const int nrb = a.R - 1, nbnd = nrb + 1 + 3 + 7;
    for (int v = tid; v < nbnd * a.El; v += NTH) {
      const int bi = v / a.El, le = v % a.El;
      long long b;
      int ki = 0, q = 0;
      if (bi < nrb) {
        b = (long long)(bi + 1) * a.Tr;
      } else {
        const int c = bi - nrb;  // 0: K = 2, q = 1; 1..3: K = 4, q = 1..3; 4..10: K = 8, q = 1..7
        ki = c < 1 ? 1 : (c < 4 ? 2 : 3);
        const int K = kopt_value(ki);
        q = c - (ki == 1 ? 0 : ki == 2 ? 1 : 4) + 1;
        b = ((long long)q * a.T + K - 1) / K;
      }
      if (b < t0 || b >= t1) continue;
      const int p = (int)(b - t0), pw = p / WAVE, pl = p % WAVE;
      int cnt = a.off[le] + a.blk_off[(size_t)blockIdx.x * a.El + le];
      for (int w = 0; w < pw; ++w) cnt += wc[w][le];
      cnt += __popcll(mk[pw][le] & (pl == 0 ? 0ull : (~0ull >> (64 - pl))));
      if (bi < nrb) a.rbnd[le * (a.R + 1) + bi + 1] = cnt;
      else a.sub_off[(ki * a.El + le) * SUBW + q] = cnt;
    }
  }
  int first = -1, first_le = MAX_SEG;
  if (valid) {
    for (int j = 0; j < a.k; ++j) {
      int le = le_j[j];
      int s = -1;
      if (le >= 0) {
        int pre = 0;
        for (int w = 0; w < wave; ++w) pre += wc[w][le];
        s = a.off[le] + a.blk_off[(size_t)blockIdx.x * a.El + le] + pre + r_j[j];
        a.inv[s] = g * a.k + j;
        if (le < first_le) { first_le = le; first = s; }
      }
      a.slot[(size_t)g * a.k + j] = s;
    }
    a.first_slot[g] = first;
    if (first >= 0) atomicAdd(&uq[g / a.Tr], 1);
  }
  __syncthreads();
  for (int r = tid; r < a.R; r += NTH)
    if (uq[r]) atomicAdd(&a.uniq[r], uq[r]);
}

// Rows of segment seg (local experts, then shared experts) in chunk q of
// the K-chunk option ki; so: that option's sub_off table.  A shared expert
// takes rank 0's tokens of the chunk (tokens [ceil(qT/K), ceil((q+1)T/K))).
__device__ inline int seg_chunk_rows(const TableArgs& a, const int* so, int ki, int K, int seg, int q) {
  if (seg < a.El) {
    const int* e = so + (ki * a.El + seg) * SUBW;
    return e[q + 1] - e[q];
  }
  const int t0 = (int)(((long long)q * a.T + K - 1) / K);
  const int t1 = min((int)(((long long)(q + 1) * a.T + K - 1) / K), a.Tr);
  return max(0, t1 - t0);
}

// One workgroup: per-(expert, rank) counts from the rank-boundary slots,
// the row map and the tile counts of the cost model from the chunk offsets,
// and the stats words.
__global__ void __launch_bounds__(NTH) tab_finalize_kernel(TableArgs a) {
  __shared__ int ntk[KOPT];
  __shared__ int xl_s;
  __shared__ int so_l[KOPT * MAX_EL * SUBW];   // this workgroup's copy of sub_off
  const int tid = threadIdx.x;
  if (tid < KOPT) ntk[tid] = 0;
  if (tid == 0) xl_s = 0;
  for (int v = tid; v < KOPT * a.El * SUBW; v += NTH) so_l[v] = a.sub_off[v];
  __syncthreads();
  for (int v = tid; v < a.El * a.R; v += NTH) {
    const int le = v / a.R, r = v % a.R;
    const int c = a.rbnd[le * (a.R + 1) + r + 1] - a.rbnd[le * (a.R + 1) + r];
    a.cnt_rank[v] = c;
    if (r == 0) atomicAdd(&xl_s, c);
  }
  // The row map (common.h): for each chunk option, the (segment, chunk)
  // pairs in segment-major order, each taking its rows rounded up to a
  // 32-row group; wavefront ki scans option ki.  Entries q >= K are zero.
  static_assert(NTH / WAVE == KOPT, "one wavefront per chunk option");
  {
    const int lane = tid & (WAVE - 1), ki = tid / WAVE, K = kopt_value(ki);
    const int nseg = a.El + a.S, n = nseg * K;
    int carry = 0;
    for (int b = 0; b < n; b += WAVE) {
      const int v = b + lane;
      const int seg = v / K, q = v - seg * K;
      const int sz = v < n ? align_rows(seg_chunk_rows(a, so_l, ki, K, seg, q)) : 0;
      int x = sz;
#pragma unroll
      for (int d = 1; d < WAVE; d <<= 1) {
        const int y = __shfl_up(x, d, WAVE);
        if (lane >= d) x += y;
      }
      if (v < n) a.row_off[(ki * nseg + seg) * SUBW + q] = carry + x - sz;
      carry += __shfl(x, WAVE - 1, WAVE);
    }
    for (int v = lane; v < nseg * (SUBW - K); v += WAVE)
      a.row_off[(ki * nseg + v / (SUBW - K)) * SUBW + K + v % (SUBW - K)] = 0;
  }
  // GEMM tiles of the layer at each chunk option: every (chunk, segment)
  // contributes ceil(rows / BM) row tiles of GEMM0 + GEMM1 tiles; shared
  // experts take rank 0's tokens of the chunk
  for (int ki = 0; ki < KOPT; ++ki) {
    const int K = kopt_value(ki), nseg = a.El + a.S;
    int part = 0;
    for (int v = tid; v < K * nseg; v += NTH) {
      const int q = v / nseg, seg = v % nseg;
      const int rows = seg_chunk_rows(a, so_l, ki, K, seg, q);
      part += (rows + BM - 1) / BM * a.tiles_per_row_tile;
    }
    if (part) atomicAdd(&ntk[ki], part);
  }
  __syncthreads();
  if (tid == 0) {
    const int X = a.off[a.El];
    int uin = 0;
    for (int r = 1; r < a.R; ++r) uin += a.uniq[r];
    a.stats[ST_X] = X;
    a.stats[ST_XLOCAL] = xl_s;
    a.stats[ST_XIN] = X - xl_s;
    a.stats[ST_ULOCAL] = a.uniq[0];
    a.stats[ST_UIN] = uin;
    for (int ki = 0; ki < KOPT; ++ki) a.stats[ST_NTK + ki] = ntk[ki];
  }
}

__global__ void zero_i32_kernel(int* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// ---------------------------------------------------------------------------
// Weight packing (one-off, not part of the layer): transposes each expert's
// [H][F] / [F][H] matrix into the slab-tiled GEMM B layout (common.h).
// W1/W3 go to [2F][H] with 32-column groups interleaved (gate f..f+31, then
// up f..f+31), so one 64-column slice of GEMM0 holds matching gate and up
// columns; W2 goes to [H][F].  pack_pad_kernel zeroes the slab padding.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(NTH) pack_transpose_kernel(PackArgs a) {
  __shared__ uint16_t tile[32][33];
  const int seg = blockIdx.z;
  const uint16_t* src = a.src + (size_t)seg * a.rows * a.cols;
  uint16_t* dst = a.dst + (size_t)seg * a.seg_stride;
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int i = ty; i < 32; i += 8) {
    int r = r0 + i, c = c0 + tx;
    if (r < a.rows && c < a.cols) tile[i][tx] = src[(size_t)r * a.cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    int c = c0 + i, r = r0 + tx;  // dst row index is the source column
    if (r < a.rows && c < a.cols) {
      int drow = a.interleave ? (c / 32) * 64 + a.which * 32 + (c % 32) : c;
      dst[slab_index(drow, r, a.rows)] = tile[tx][i];
    }
  }
}

__global__ void __launch_bounds__(NTH) pack_pad_kernel(PadArgs a) {
  const int pad = (int)(slab_rows(a.R) - a.R);
  const long long per_seg = (long long)pad * a.K;
  for (long long v = (long long)blockIdx.x * NTH + threadIdx.x; v < per_seg * a.nseg; v += (long long)gridDim.x * NTH) {
    const int seg = (int)(v / per_seg);
    const long long e = v - seg * per_seg;
    const int n = a.R + (int)(e / a.K), k = (int)(e % a.K);
    a.dst[seg * a.seg_stride + slab_index(n, k, a.K)] = 0;
  }
}

}  // namespace moe
