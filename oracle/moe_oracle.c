/*
 * CPU oracle for one GPU's share of an expert-parallel MoE layer.
 * TEST INFRASTRUCTURE ONLY: see moe_oracle.h.  Built with -O2, no fast-math,
 * no FP contraction, single thread.
 */
#include "moe_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static float bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* ---- routing (input of the MoE layer, section 4) ---------------------- */

void orc_gate_logits(const uint16_t* x, const uint16_t* wg, const float* bias,
                     int T, int H, int E, float* logits) {
  float* acc = (float*)malloc(sizeof(float) * (size_t)(E > 0 ? E : 1));
  for (int g = 0; g < T; ++g) {
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;
    const uint16_t* xr = x + (size_t)g * H;
    for (int h = 0; h < H; ++h) {
      float xv = bf16_to_f32(xr[h]);
      const uint16_t* wr = wg + (size_t)h * E;
      for (int e = 0; e < E; ++e) acc[e] = acc[e] + xv * bf16_to_f32(wr[e]);
    }
    for (int e = 0; e < E; ++e)
      logits[(size_t)g * E + e] = bias ? acc[e] + bias[e] : acc[e];
  }
  free(acc);
}

void orc_softmax_topk(const float* logits, int T, int E, int k, int32_t* idx, double* w) {
  double* p = (double*)malloc(sizeof(double) * (size_t)E);
  char* taken = (char*)malloc((size_t)E);
  for (int g = 0; g < T; ++g) {
    const float* l = logits + (size_t)g * E;
    /* softmax over all experts */
    double m = l[0];
    for (int e = 1; e < E; ++e) if (l[e] > m) m = l[e];
    double z = 0.0;
    for (int e = 0; e < E; ++e) { p[e] = exp((double)l[e] - m); z += p[e]; }
    for (int e = 0; e < E; ++e) p[e] /= z;
    /* top-k on the logits: larger first, equal -> smaller id */
    memset(taken, 0, (size_t)E);
    double ps = 0.0;
    for (int j = 0; j < k; ++j) {
      int best = -1;
      for (int e = 0; e < E; ++e) {
        if (taken[e]) continue;
        if (best < 0 || l[e] > l[best]) best = e;
      }
      taken[best] = 1;
      idx[(size_t)g * k + j] = best;
      ps += p[best];
    }
    /* renormalise the selected probabilities */
    for (int j = 0; j < k; ++j)
      w[(size_t)g * k + j] = p[idx[(size_t)g * k + j]] / ps;
  }
  free(p);
  free(taken);
}

/* ---- routing tables (section 3.1, section 4) --------------------------- */

int orc_route_tables(const int32_t* idx, int T, int k, int R, int Tr, int e0, int El,
                     int32_t* cnt_rank, int32_t* uniq, int32_t* off, int32_t* slot,
                     int32_t* inv, int32_t* first_slot) {
  for (int i = 0; i < El * R; ++i) cnt_rank[i] = 0;
  for (int r = 0; r < R; ++r) uniq[r] = 0;
  for (int i = 0; i < T * k; ++i) slot[i] = -1;
  for (int g = 0; g < T; ++g) first_slot[g] = -1;

  /* slots in (expert, token) order: expert le's rows are contiguous and
   * sorted by token index */
  int s = 0;
  for (int le = 0; le < El; ++le) {
    off[le] = s;
    for (int g = 0; g < T; ++g) {
      for (int j = 0; j < k; ++j) {
        if (idx[(size_t)g * k + j] - e0 == le) {
          slot[(size_t)g * k + j] = s;
          inv[s] = g * k + j;
          cnt_rank[le * R + g / Tr] += 1;
          if (first_slot[g] < 0) first_slot[g] = s;  /* le ascending: first hit is the smallest le */
          ++s;
        }
      }
    }
  }
  off[El] = s;
  for (int g = 0; g < T; ++g)
    if (first_slot[g] >= 0) uniq[g / Tr] += 1;
  return s;
}

void orc_chunk_offsets(const int32_t* inv, const int32_t* off, int T, int k, int El, int K,
                       int32_t* sub_off) {
  for (int le = 0; le < El; ++le) {
    for (int q = 0; q <= K; ++q) {
      /* first slot of expert le whose token has chunk >= q */
      int s = off[le];
      while (s < off[le + 1]) {
        int g = inv[s] / k;
        long long chunk = ((long long)g * K) / T;
        if (chunk >= q) break;
        ++s;
      }
      sub_off[le * (K + 1) + q] = s;
    }
  }
}

void orc_dispatch(const uint16_t* x, const int32_t* inv, int X, int k, int H, uint16_t* A) {
  for (int s = 0; s < X; ++s) {
    int g = inv[s] / k;
    memcpy(A + (size_t)s * H, x + (size_t)g * H, sizeof(uint16_t) * (size_t)H);
  }
}

/* ---- expert FFN and combine (section 2.1, Fig 3) ----------------------- */

void orc_expert_ffn(const uint16_t* a, const uint16_t* w1, const uint16_t* w3,
                    const uint16_t* w2, int H, int F, double* out) {
  double* u1 = (double*)calloc((size_t)F, sizeof(double));
  double* u3 = (double*)calloc((size_t)F, sizeof(double));
  /* GEMM0: gate (W1) and up (W3) projections */
  for (int h = 0; h < H; ++h) {
    double av = bf16_to_f32(a[h]);
    const uint16_t* r1 = w1 + (size_t)h * F;
    const uint16_t* r3 = w3 + (size_t)h * F;
    for (int f = 0; f < F; ++f) {
      u1[f] += av * (double)bf16_to_f32(r1[f]);
      u3[f] += av * (double)bf16_to_f32(r3[f]);
    }
  }
  /* activation: SiLU of the gate times the up projection */
  for (int f = 0; f < F; ++f) {
    double z = u1[f];
    u1[f] = (z / (1.0 + exp(-z))) * u3[f];
  }
  /* GEMM1: down projection */
  for (int h = 0; h < H; ++h) out[h] = 0.0;
  for (int f = 0; f < F; ++f) {
    double hv = u1[f];
    const uint16_t* r2 = w2 + (size_t)f * H;
    for (int h = 0; h < H; ++h) out[h] += hv * (double)bf16_to_f32(r2[h]);
  }
  free(u1);
  free(u3);
}

void orc_layer_rows(const uint16_t* x, const int32_t* idx, const double* w,
                    const uint16_t* w1, const uint16_t* w3, const uint16_t* w2,
                    const uint16_t* ws1, const uint16_t* ws3, const uint16_t* ws2,
                    int k, int Tr, int H, int F, int e0, int El, int S,
                    const int64_t* rows, int n_rows, double* y) {
  double* o = (double*)malloc(sizeof(double) * (size_t)H);
  const size_t ew = (size_t)H * F;
  for (int i = 0; i < n_rows; ++i) {
    int64_t g = rows[i];
    const uint16_t* xr = x + (size_t)g * H;
    double* yr = y + (size_t)i * H;
    for (int h = 0; h < H; ++h) yr[h] = 0.0;
    for (int j = 0; j < k; ++j) {
      int le = idx[g * k + j] - e0;
      if (le < 0 || le >= El) continue;
      orc_expert_ffn(xr, w1 + le * ew, w3 + le * ew, w2 + le * ew, H, F, o);
      double wj = w[g * k + j];
      for (int h = 0; h < H; ++h) yr[h] += wj * o[h];
    }
    if (g < Tr) {
      for (int s = 0; s < S; ++s) {
        orc_expert_ffn(xr, ws1 + s * ew, ws3 + s * ew, ws2 + s * ew, H, F, o);
        for (int h = 0; h < H; ++h) yr[h] += o[h];
      }
    }
  }
  free(o);
}

/* ---- cost model (sections 3.1-3.3) ------------------------------------- */

int64_t orc_tile_count(const int32_t* rows_seg, int n_seg, int K, int BM, int nt0, int nt1) {
  int64_t n = 0;
  for (int seg = 0; seg < n_seg; ++seg)
    for (int q = 0; q < K; ++q) {
      int64_t m = rows_seg[seg * K + q];
      int64_t mt = (m + BM - 1) / BM;
      n += mt * (int64_t)(nt0 + nt1);
    }
  return n;
}

double orc_t_total(const orc_plan_in* in, int ci, int ki) {
  double bw = in->bw[ci];
  double fl = in->flops[ci];
  double eff = in->eff[ki];
  double K = (double)in->K[ki];
  double t_comp = in->w_comp / (fl * eff);                              /* Eq 9 */
  double t_comm = (in->w_dispatch + in->w_combine) / bw;                /* Eq 5 */
  double bw_tail = in->bw_all > 0.0 ? in->bw_all : bw;
  double t_tail = ((1.0 - in->alpha) * in->w_combine) / (bw_tail * K);  /* Eq 10 */
  double a = t_comp + t_tail;
  return a > t_comm ? a : t_comm;                                       /* Eq 15 */
}

void orc_plan(const orc_plan_in* in, orc_plan_out* out) {
  int bc = 0, bk = 0;
  double best = orc_t_total(in, 0, 0);
  for (int ci = 0; ci < in->n_c; ++ci)
    for (int ki = 0; ki < in->n_k; ++ki) {
      double t = orc_t_total(in, ci, ki);
      if (t < best) { best = t; bc = ci; bk = ki; }                    /* Eq 16 */
    }
  out->ci = bc;
  out->ki = bk;
  out->c = in->c[bc];
  out->K = in->K[bk];
  out->t_total = best;
  /* bubble stealing at (c*, K*).  Eq 11's communication volume, read as
   * selected by steal_window (see moe_oracle.h): the plain reading takes the
   * whole movement volume of Eq 5; the others leave out what every worker
   * moves outside the window (the last chunk's combine, section 4, and under
   * movement stealing the first chunk's dispatch). */
  double kd = (double)in->K[bk];
  double w_win;
  if (in->steal_window == 1)
    w_win = ((in->w_dispatch + in->w_combine) * (kd - 1.0)) / kd;
  else if (in->steal_window == 2)
    w_win = in->w_dispatch + (in->w_combine * (kd - 1.0)) / kd;
  else
    w_win = in->w_dispatch + in->w_combine;
  double t_comm = w_win / in->bw[bc];                                  /* Eq 11 */
  double w_partial = t_comm * in->flops[bc];                           /* Eq 12 */
  double w_steal = in->w_comp - w_partial;                             /* Eq 13 */
  if (w_steal < 0.0) w_steal = 0.0;
  int64_t nt = in->n_tiles[bk];
  int n_steal = 0;
  if (nt > 0 && in->w_comp > 0.0) {
    double w_tile = in->w_comp / (double)nt;
    double share = w_steal / ((double)in->N * w_tile);                 /* Eq 14 */
    n_steal = (int)(in->steal_ceil ? ceil(share) : floor(share));
  }
  out->n_steal = n_steal;
}
