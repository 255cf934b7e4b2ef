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
constexpr int GEPL = MAX_E / GG;  // experts per lane
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

// Candidates of the GTOK tokens from g0 on (one workgroup of NTH threads):
// tau = k-th largest lower end; every expert whose upper end reaches tau
// becomes a chain (g, e) of the chain list, in expert order per token.  The
// workgroup takes its chain range with one atomic.
__device__ __forceinline__ void cand_tokens(const GateArgs& a, int g0, int* cnt, int& base_s) {
  const int tid = threadIdx.x, grp = tid / GG, gl = tid % GG;
  const int g = g0 + grp;
  const bool valid = g < a.T;
  const int gs = valid ? g : 0;
  const float xn = a.xn[gs];
  float lo[GEPL], hi[GEPL];
#pragma unroll
  for (int i = 0; i < GEPL; ++i) {
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
    for (int i = 0; i < GEPL; ++i)
      if (better(lo[i], gl + GG * i, v, e)) { v = lo[i]; e = gl + GG * i; }
    group_argmax(v, e);
    tau = v;
#pragma unroll
    for (int i = 0; i < GEPL; ++i)
      if (gl + GG * i == e) lo[i] = -INFINITY;
  }
  int mine = 0;
#pragma unroll
  for (int i = 0; i < GEPL; ++i) mine += valid && hi[i] >= tau;
  int pre = mine;
#pragma unroll
  for (int d = 1; d < GG; d <<= 1) {
    const int o = __shfl_up(pre, d, GG);
    if (gl >= d) pre += o;
  }
  const int total = __shfl(pre, GG - 1, GG);
  if (gl == 0) cnt[grp] = total;
  __syncthreads();
  if (tid == 0) {
    int t = 0;
    for (int q = 0; q < GTOK; ++q) { const int c = cnt[q]; cnt[q] = t; t += c; }
    base_s = atomicAdd(&a.stats[ST_CANDS], t);
  }
  __syncthreads();
  const int tb = base_s + cnt[grp];
  if (valid && gl == 0) {
    a.tok_base[g] = tb;
    a.tok_n[g] = total;
  }
  // this lane's candidates, in expert order within the lane; the final pass
  // does not depend on the order
  int pos = tb + pre - mine;
#pragma unroll
  for (int i = 0; i < GEPL; ++i)
    if (valid && hi[i] >= tau) {
      a.ch_g[pos] = g;
      a.ch_e[pos] = gl + GG * i;
      ++pos;
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
  __shared__ int cnt[GTOK];
  __shared__ int base_s;
  __shared__ float red[GATE_WAVES - 1][32 * 32 * 4];
  __shared__ float ssr[GATE_WAVES][64];
  __shared__ __align__(16) char ring[GATE_WAVES * GS_ST * GS_SB];
  if (a.E <= 32 && (a.H / GATE_WAVES) % 64 == 0) gate_mfma_staged(a, ring, red, ssr);
  else if (a.E <= 32) gate_mfma_body<1, 8, GATE_WAVES>(a, red, ssr);
  else gate_mfma_body<4, 4, GATE_WAVES>(a, red, ssr);
  __syncthreads();
  for (int sub = 0; sub < 32 / GTOK; ++sub) {
    cand_tokens(a, blockIdx.x * 32 + sub * GTOK, cnt, base_s);
    __syncthreads();
  }
}

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

// top-k of the candidates' defined logits (descending, equal logits ->
// smaller id); softmax normaliser from the defined logits of the candidates
// and the approximate ones elsewhere (it cancels in the renormalisation)
__global__ void __launch_bounds__(NTH) gate_final_kernel(GateArgs a) {
  __shared__ uint32_t cmask[GTOK][MAX_E / 32];
  const int tid = threadIdx.x, grp = tid / GG, gl = tid % GG;
  const int g = blockIdx.x * GTOK + grp;
  const bool valid = g < a.T;
  const int gs = valid ? g : 0;
  for (int i = gl; i < MAX_E / 32; i += GG) cmask[grp][i] = 0u;
  __builtin_amdgcn_wave_barrier();
  const int tb = valid ? a.tok_base[g] : 0, tn = valid ? a.tok_n[g] : 0;
  for (int c = gl; c < tn; c += GG) {
    const int e = a.ch_e[tb + c];
    atomicOr(&cmask[grp][e >> 5], 1u << (e & 31));
  }
  __builtin_amdgcn_wave_barrier();
  float tv[MAX_TOPK];
  int ti[MAX_TOPK];
  for (int r = 0; r < a.k; ++r) {
    float v = -INFINITY;
    int e = 1 << 30;
    for (int c = gl; c < tn; c += GG) {
      const int ce = a.ch_e[tb + c];
      const float cv = a.ch_l[tb + c];
      bool taken = false;
      for (int q = 0; q < r; ++q) taken |= ti[q] == ce;
      if (!taken && better(cv, ce, v, e)) { v = cv; e = ce; }
    }
    group_argmax(v, e);
    tv[r] = v;
    ti[r] = e;
  }
  const float m = tv[0];
  const float xn = a.xn[gs];
  float z = 0.0f;
#pragma unroll
  for (int i = 0; i < GEPL; ++i) {
    const int e = gl + GG * i;
    if (e < a.E && !((cmask[grp][e >> 5] >> (e & 31)) & 1u)) {
      float l, d;
      interval(a, gs, e, xn, l, d);
      z += expf(l - m);
    }
  }
  for (int c = gl; c < tn; c += GG) z += expf(a.ch_l[tb + c] - m);
#pragma unroll
  for (int d = GG / 2; d > 0; d >>= 1) z += __shfl_xor(z, d, WAVE);
  if (gl == 0 && valid) {
    float p[MAX_TOPK];
    float ps = 0.0f;
    for (int j = 0; j < a.k; ++j) { p[j] = expf(tv[j] - m) / z; ps += p[j]; }
    for (int j = 0; j < a.k; ++j) {
      a.topk_idx[(size_t)g * a.k + j] = ti[j];
      a.topk_w[(size_t)g * a.k + j] = p[j] / ps;
    }
  }
}

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

__global__ void __launch_bounds__(NTH) tab_count_kernel(TableArgs a) {
  __shared__ int hist[MAX_SEG];
  __shared__ int nbad;
  const int tid = threadIdx.x;
  for (int i = tid; i < a.El; i += NTH) hist[i] = 0;
  if (tid == 0) nbad = 0;
  __syncthreads();
  const int g = blockIdx.x * TB + tid;
  bool bad = false;
  if (g < a.T) {
    int ids[MAX_TOPK];
    for (int j = 0; j < a.k; ++j) ids[j] = a.topk_idx[(size_t)g * a.k + j];
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

__global__ void __launch_bounds__(NTH) tab_scan_kernel(TableArgs a) {
  __shared__ int tot[MAX_SEG];
  const int tid = threadIdx.x;
  for (int le = tid; le < a.El; le += NTH) {
    int run = 0;
    for (int b = 0; b < a.nblk; ++b) {
      int c = a.blk_cnt[(size_t)b * a.El + le];
      a.blk_off[(size_t)b * a.El + le] = run;
      run += c;
    }
    tot[le] = run;
  }
  __syncthreads();
  if (tid == 0) {
    int s = 0;
    for (int le = 0; le < a.El; ++le) { a.off[le] = s; s += tot[le]; }
    a.off[a.El] = s;
    // the table builder's stats words: the bad-id count here, the rest in
    // tab_finalize (words it does not write stay zero)
    int bad = 0;
    for (int b = 0; b < a.nblk; ++b) bad += a.blk_bad[b];
    for (int w = 0; w < ST_CANDS; ++w) a.stats[w] = w == ST_BADIDS ? bad : 0;
  }
}

__global__ void __launch_bounds__(NTH) tab_perm_kernel(TableArgs a) {
  __shared__ int wc[NTH / WAVE][MAX_SEG];
  const int tid = threadIdx.x;
  const int lane = tid & (WAVE - 1);
  const int wave = tid / WAVE;
  const int g = blockIdx.x * TB + tid;
  const bool valid = g < a.T;

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
    if (lane == 0) wc[wave][le] = __popcll(m);
  }
  __syncthreads();
  if (!valid) return;
  int first = -1, first_le = MAX_SEG;
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
}

// Lower bounds in an expert's segment of slots (tokens ascending): the first
// slot of expert le whose token is >= b.  The workgroup first stages the
// token of every STRIDE-th slot in LDS (samp); a search narrows to one
// window of STRIDE slots there and finishes with a binary search of
// log2(STRIDE) global reads.
constexpr int FIN_SAMP = 4096;
__device__ inline int slot_token(const TableArgs& a, int p) { return a.inv[p] / a.k; }
__device__ inline int seg_lower_bound(const TableArgs& a, const int* samp, int stride, int le, long long b) {
  int lo = a.off[le], hi = a.off[le + 1];
  int jlo = (lo + stride - 1) / stride, jhi = (hi + stride - 1) / stride;  // samples at slots in [lo, hi)
  int j0 = jlo, j1 = jhi;
  while (j0 < j1) {  // first sample whose token is >= b
    const int mid = (j0 + j1) >> 1;
    if ((long long)samp[mid] < b) j0 = mid + 1; else j1 = mid;
  }
  if (j0 > jlo) lo = (j0 - 1) * stride + 1;  // the sample before has a token < b
  if (j0 < jhi) hi = j0 * stride;            // this sample has a token >= b
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if ((long long)slot_token(a, mid) < b) lo = mid + 1; else hi = mid;
  }
  return lo;
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

// One workgroup.  Lower bounds at the rank boundaries (per-(expert, rank)
// counts) and at the chunk boundaries of every chunk option (sub_off) form
// one item space, one search per item and thread; the row map and the tile
// counts of the cost model are then taken from the workgroup's copy of
// sub_off.
__global__ void __launch_bounds__(NTH) tab_finalize_kernel(TableArgs a) {
  __shared__ int uq[64];
  __shared__ int ntk[KOPT];
  __shared__ int samp[FIN_SAMP];
  __shared__ int rb[MAX_EL * 65];              // [El][R + 1] lower bounds at rank boundaries
  __shared__ int so_l[KOPT * MAX_EL * SUBW];   // this workgroup's copy of sub_off
  const int tid = threadIdx.x;
  const int X = a.off[a.El];
  int stride = 64;
  while ((X + stride - 1) / stride > FIN_SAMP) stride *= 2;
  for (int r = tid; r < a.R; r += NTH) uq[r] = 0;
  if (tid < KOPT) ntk[tid] = 0;
  for (int j = tid; j * stride < X; j += NTH) samp[j] = slot_token(a, j * stride);
  __syncthreads();
  // unique tokens per rank (tokens with at least one local pair)
  for (int g = tid; g < a.T; g += NTH)
    if (a.first_slot[g] >= 0) atomicAdd(&uq[g / a.Tr], 1);
  const int n_rank = a.El * (a.R + 1), n_sub = KOPT * a.El * SUBW;
  for (int v = tid; v < n_rank + n_sub; v += NTH) {
    if (v < n_rank) {
      // rank r owns tokens [r*Tr, (r+1)*Tr)
      const int le = v / (a.R + 1), r = v % (a.R + 1);
      rb[v] = seg_lower_bound(a, samp, stride, le, (long long)r * a.Tr);
    } else {
      // chunk offsets: chunk(g) = floor(g*K/T) >= q  <=>  g >= ceil(q*T/K)
      const int w = v - n_rank;
      const int ki = w / (a.El * SUBW), rem = w % (a.El * SUBW);
      const int le = rem / SUBW, q = rem % SUBW;
      const int K = kopt_value(ki);
      int val = 0;
      if (q <= K) val = seg_lower_bound(a, samp, stride, le, ((long long)q * a.T + K - 1) / K);
      a.sub_off[w] = val;
      so_l[w] = val;
    }
  }
  __syncthreads();
  for (int v = tid; v < a.El * a.R; v += NTH) {
    const int le = v / a.R, r = v % a.R;
    a.cnt_rank[v] = rb[le * (a.R + 1) + r + 1] - rb[le * (a.R + 1) + r];
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
  for (int r = tid; r < a.R; r += NTH) a.uniq[r] = uq[r];
  if (tid == 0) {
    int xl = 0;
    for (int le = 0; le < a.El; ++le) xl += rb[le * (a.R + 1) + 1] - rb[le * (a.R + 1)];
    int uin = 0;
    for (int r = 1; r < a.R; ++r) uin += uq[r];
    a.stats[ST_X] = X;
    a.stats[ST_XLOCAL] = xl;
    a.stats[ST_XIN] = X - xl;
    a.stats[ST_ULOCAL] = uq[0];
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
