// Routing that precedes the MoE layer (the layer takes the routing result as
// its input, paper section 4) and the routing tables of this GPU's share
// (section 3.1 descriptors X_local, X_in, X_in^uniq; the dispatch permutation
// and its deduplication, section 4; the chunk offsets of section 3.2.1).
//
// Everything here is deterministic: logits use one fp32 accumulator per
// (token, expert) over ascending h, and slots come from block histograms, an
// ordered scan and wavefront ballots, never from atomic slot claiming.
#include "common.h"
#include "kernels.h"

namespace moe {

// ---------------------------------------------------------------------------
// Gate: logits -> softmax -> top-k (on logits, ties -> smaller id) -> renormalise
// Each thread owns a TPT-token x EPT-expert block of logits (one fp32
// accumulator per (token, expert), ascending h).  x and Wg are staged
// through LDS as fp32 in chunks of GH hidden values, token-major and
// expert-major rows padded to GHP floats so float4 reads are conflict-free.
// The host picks the block size so that the grid has enough workgroups.
// ---------------------------------------------------------------------------
constexpr int GH = 16;
constexpr int GHP = GH + 4;
constexpr int GATE_MAX_TT = 256;

template <int TPT, int EPT>
__global__ void __launch_bounds__(NTH) gate_topk_kernel(GateArgs a) {
  __shared__ __attribute__((aligned(16))) float xs[GATE_MAX_TT * GHP];
  __shared__ __attribute__((aligned(16))) float ws[MAX_E * GHP];
  __shared__ float lg[NTH * 16];

  const int tid = threadIdx.x;
  const int EQ = (a.E + EPT - 1) / EPT;
  const int EP = EQ * EPT;
  const int TQ = a.tq;  // token groups per workgroup
  const int TT = TQ * TPT;
  const int g0 = blockIdx.x * TT;
  const bool active = tid < TQ * EQ;
  const int tq = active ? tid / EQ : 0;
  const int eq = active ? tid % EQ : 0;

  float acc[TPT][EPT];
#pragma unroll
  for (int i = 0; i < TPT; ++i)
#pragma unroll
    for (int j = 0; j < EPT; ++j) acc[i][j] = 0.0f;

  for (int h0 = 0; h0 < a.H; h0 += GH) {
    // stage x[g0 .. g0+TT)[h0 .. h0+GH) as xs[t][h]
    for (int v = tid; v < TT * (GH / 8); v += NTH) {
      const int t = v / (GH / 8), part = v % (GH / 8);
      const int g = g0 + t;
      u32x4_t w = {0u, 0u, 0u, 0u};
      if (g < a.T) w = *reinterpret_cast<const u32x4_t*>(a.x + (size_t)g * a.H + h0 + part * 8);
      float* d = xs + t * GHP + part * 8;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        d[2 * q] = bf16_lo(w[q]);
        d[2 * q + 1] = bf16_hi(w[q]);
      }
    }
    // stage Wg[h0 .. h0+GH)[0 .. E) as ws[e][h]
    for (int v = tid; v < GH * EP; v += NTH) {
      const int h = v / EP, e = v % EP;
      ws[e * GHP + h] = e < a.E ? bf16_to_f32(a.wg[(size_t)(h0 + h) * a.E + e]) : 0.0f;
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int h = 0; h < GH; h += 4) {
        float4 xv[TPT], wv[EPT];
#pragma unroll
        for (int i = 0; i < TPT; ++i) xv[i] = *reinterpret_cast<const float4*>(xs + (tq * TPT + i) * GHP + h);
#pragma unroll
        for (int j = 0; j < EPT; ++j) wv[j] = *reinterpret_cast<const float4*>(ws + (eq * EPT + j) * GHP + h);
        // products of two bf16 values are exact in fp32, so a fused or an
        // unfused multiply-add gives the same rounded sum; h ascends
#pragma unroll
        for (int i = 0; i < TPT; ++i)
#pragma unroll
          for (int j = 0; j < EPT; ++j) {
            acc[i][j] = acc[i][j] + xv[i].x * wv[j].x;
            acc[i][j] = acc[i][j] + xv[i].y * wv[j].y;
            acc[i][j] = acc[i][j] + xv[i].z * wv[j].z;
            acc[i][j] = acc[i][j] + xv[i].w * wv[j].w;
          }
      }
    }
    __syncthreads();
  }

  if (active) {
#pragma unroll
    for (int i = 0; i < TPT; ++i)
#pragma unroll
      for (int j = 0; j < EPT; ++j) {
        const int e = eq * EPT + j;
        if (e < a.E) {
          float l = acc[i][j];
          if (a.bias) l = l + a.bias[e];
          lg[(tq * TPT + i) * EP + e] = l;
        }
      }
  }
  __syncthreads();

  // one thread per token: softmax statistics, top-k insertion, renormalise
  for (int t = tid; t < TT; t += NTH) {
    const int g = g0 + t;
    if (g >= a.T) break;
    const float* l = lg + t * EP;
    float m = l[0];
    for (int e = 1; e < a.E; ++e) m = fmaxf(m, l[e]);
    float z = 0.0f;
    for (int e = 0; e < a.E; ++e) z += expf(l[e] - m);

    float tv[MAX_TOPK];
    int ti[MAX_TOPK];
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j) { tv[j] = -INFINITY; ti[j] = -1; }
    for (int e = 0; e < a.E; ++e) {
      const float v = l[e];
      // insert e if it beats the current k-th entry; equal logits keep the
      // earlier (smaller) expert id in front
      if (ti[a.k - 1] >= 0 && !(v > tv[a.k - 1])) continue;
      int carry_i = e;
      float carry_v = v;
      bool placed = false;
#pragma unroll
      for (int j = 0; j < MAX_TOPK; ++j) {
        if (j < a.k) {
          const bool go = placed || ti[j] < 0 || carry_v > tv[j];
          if (go) {
            const float sv = tv[j];
            const int si = ti[j];
            tv[j] = carry_v;
            ti[j] = carry_i;
            carry_v = sv;
            carry_i = si;
            placed = true;
            if (si < 0) break;
          }
        }
      }
    }
    float p[MAX_TOPK];
    float ps = 0.0f;
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j)
      if (j < a.k) { p[j] = expf(tv[j] - m) / z; ps += p[j]; }
#pragma unroll
    for (int j = 0; j < MAX_TOPK; ++j)
      if (j < a.k) {
        a.topk_idx[(size_t)g * a.k + j] = ti[j];
        a.topk_w[(size_t)g * a.k + j] = p[j] / ps;
      }
  }
}

template __global__ void gate_topk_kernel<4, 4>(GateArgs);
template __global__ void gate_topk_kernel<2, 2>(GateArgs);
template __global__ void gate_topk_kernel<1, 1>(GateArgs);

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
  const int tid = threadIdx.x;
  for (int i = tid; i < a.El; i += NTH) hist[i] = 0;
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
    atomicAdd(&a.stats[ST_BADIDS], 1);
    atomicOr(a.err, ERR_ROUTING);
  }
  __syncthreads();
  for (int i = tid; i < a.El; i += NTH) a.blk_cnt[(size_t)blockIdx.x * a.El + i] = hist[i];
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

// first slot of expert le whose token index is >= b (segment is sorted by token)
__device__ inline int seg_lower_bound(const TableArgs& a, int le, long long b) {
  int lo = a.off[le], hi = a.off[le + 1];
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if ((long long)(a.inv[mid] / a.k) < b) lo = mid + 1; else hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(NTH) tab_finalize_kernel(TableArgs a) {
  __shared__ int uq[64];
  const int tid = threadIdx.x;
  for (int r = tid; r < a.R; r += NTH) uq[r] = 0;
  __syncthreads();
  // per-(expert, rank) counts: rank r owns tokens [r*Tr, (r+1)*Tr)
  for (int v = tid; v < a.El * a.R; v += NTH) {
    int le = v / a.R, r = v % a.R;
    a.cnt_rank[v] = seg_lower_bound(a, le, (long long)(r + 1) * a.Tr) -
                    seg_lower_bound(a, le, (long long)r * a.Tr);
  }
  // chunk offsets: chunk(g) = floor(g*K/T) >= q  <=>  g >= ceil(q*T/K)
  for (int v = tid; v < KOPT * a.El * SUBW; v += NTH) {
    int ki = v / (a.El * SUBW);
    int rem = v % (a.El * SUBW);
    int le = rem / SUBW, q = rem % SUBW;
    int K = kopt_value(ki);
    int val = 0;
    if (q <= K) {
      long long b = ((long long)q * a.T + K - 1) / K;
      val = seg_lower_bound(a, le, b);
    }
    a.sub_off[v] = val;
  }
  // unique tokens per rank (tokens with at least one local pair)
  for (int g = tid; g < a.T; g += NTH)
    if (a.first_slot[g] >= 0) atomicAdd(&uq[g / a.Tr], 1);
  __syncthreads();
  for (int r = tid; r < a.R; r += NTH) a.uniq[r] = uq[r];
  __syncthreads();
  if (tid == 0) {
    int X = a.off[a.El];
    int xl = 0;
    for (int le = 0; le < a.El; ++le) xl += a.cnt_rank[le * a.R + 0];
    int uin = 0;
    for (int r = 1; r < a.R; ++r) uin += uq[r];
    a.stats[ST_X] = X;
    a.stats[ST_XLOCAL] = xl;
    a.stats[ST_XIN] = X - xl;
    a.stats[ST_ULOCAL] = uq[0];
    a.stats[ST_UIN] = uin;
  }
}

__global__ void zero_i32_kernel(int* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// ---------------------------------------------------------------------------
// Weight packing (one-off, not part of the layer): transposes each expert's
// [H][F] / [F][H] matrix into the k-contiguous GEMM operand layout.
// W1/W3 go to [2F][H] with 32-column groups interleaved (gate f..f+31, then
// up f..f+31), so one 64-column slice of GEMM0 holds matching gate and up
// columns; W2 goes to [H][F].
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
      dst[(size_t)drow * a.rows + r] = tile[tx][i];
    }
  }
}

}  // namespace moe
