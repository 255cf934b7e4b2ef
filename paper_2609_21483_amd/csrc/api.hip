// Host side of the C ABI declared in include/moe.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "common.h"
#include "kernels.h"

using namespace moe;

namespace {

thread_local std::string g_err;

moe_status fail(moe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(MOE_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

namespace {

// The gate's scratch: everything its kernels use besides their inputs and
// outputs (the transposed gate matrix and its row norms, the approximate
// logits and token norms, the candidate chains and their exact logits, each
// token's range of chains, and the chain counter in stats word ST_CANDS).
struct GateLayout {
  size_t wgt, lt, xn, wn, chg, che, chl, tb, tn, stats, total;
};
GateLayout gate_layout(long long T, long long H, long long E) {
  GateLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 256); return at; };
  L.wgt = take(sizeof(uint16_t) * (size_t)(E * H));
  L.lt = take(sizeof(float) * (size_t)(T * E));
  L.xn = take(sizeof(float) * (size_t)T);
  L.wn = take(sizeof(float) * (size_t)E);
  L.chg = take(sizeof(int32_t) * (size_t)(T * E));
  L.che = take(sizeof(int32_t) * (size_t)(T * E));
  L.chl = take(sizeof(float) * (size_t)(T * E));
  L.tb = take(sizeof(int32_t) * (size_t)T);
  L.tn = take(sizeof(int32_t) * (size_t)T);
  L.stats = take(sizeof(int32_t) * ST_WORDS);
  L.total = o;
  return L;
}

// Points the gate's scratch arguments into `base` laid out by L; the chain
// counter goes to `stats` (a stats block of ST_WORDS words).
void bind_gate(GateArgs& g, char* base, const GateLayout& L, int32_t* stats) {
  g.wgt = reinterpret_cast<uint16_t*>(base + L.wgt);
  g.lt = reinterpret_cast<float*>(base + L.lt);
  g.xn = reinterpret_cast<float*>(base + L.xn);
  g.wn = reinterpret_cast<float*>(base + L.wn);
  g.ch_g = reinterpret_cast<int32_t*>(base + L.chg);
  g.ch_e = reinterpret_cast<int32_t*>(base + L.che);
  g.ch_l = reinterpret_cast<float*>(base + L.chl);
  g.tok_base = reinterpret_cast<int32_t*>(base + L.tb);
  g.tok_n = reinterpret_cast<int32_t*>(base + L.tn);
  g.stats = stats;
}

// Top-k routing (gate logits, softmax, top-k, renormalisation) on a bound
// GateArgs: the certified filter's kernels in order on `s`.  tab: the
// routing tables to start on the chosen ids (their counting step, done by the
// last kernel), or null.
moe_status launch_gate(GateArgs& g, hipStream_t s, const TableArgs* tab) {
  // |L - L~| <= (gamma_{H-1}(2^-24) + gamma_H(2^-23)) * sum_h |x_h w_h|: the
  // defined recursive fp32 sum and an fp32 accumulation of the MFMA products
  // allowed twice the unit roundoff; sum |x w| <= ||x|| ||w||; 1% for the norms
  {
    const double H = (double)g.H, u = std::ldexp(1.0, -24), u2 = std::ldexp(1.0, -23);
    const double g1 = (H - 1.0) * u / (1.0 - (H - 1.0) * u), g2 = H * u2 / (1.0 - H * u2);
    g.bound = (float)(1.01 * (g1 + g2));
  }
  gate_prep_kernel<<<g.E, NTH, 0, s>>>(g);
  if (g.E <= 32) gate_mfma_kernel<<<(g.T + 31) / 32, GATE_WAVES * WAVE, 0, s>>>(g);
  // more experts: LDS-staged tiles, 128 tokens each when that still gives
  // every CU a tile, else 64
  else if (g.E <= 128) {
    // logits and candidates without leaving LDS, 128 tokens per workgroup
    // when that still gives every CU a tile, else 64
    if (g.T >= 128 * 256) gate_tile2_kernel<128><<<(g.T + 127) / 128, 2 * NTH, 0, s>>>(g);
    else gate_tile2_kernel<64><<<(g.T + 63) / 64, 2 * NTH, 0, s>>>(g);
  } else {
    // experts per lane of the candidate pass (16 lanes per token)
    const int epl = g.E <= 64 ? 4 : g.E <= 128 ? 8 : 32;
    const bool big = g.T >= 128 * 256;
    const dim3 grid(big ? (g.T + 127) / 128 : (g.T + 63) / 64);
    if (big) {
      if (epl == 4) gate_tile_kernel<128, 4><<<grid, NTH, 0, s>>>(g);
      else if (epl == 8) gate_tile_kernel<128, 8><<<grid, NTH, 0, s>>>(g);
      else gate_tile_kernel<128, 32><<<grid, NTH, 0, s>>>(g);
    } else {
      if (epl == 4) gate_tile_kernel<64, 4><<<grid, NTH, 0, s>>>(g);
      else if (epl == 8) gate_tile_kernel<64, 8><<<grid, NTH, 0, s>>>(g);
      else gate_tile_kernel<64, 32><<<grid, NTH, 0, s>>>(g);
    }
  }
  if (g.E <= 128 && g.k >= 4 && (long long)g.T * g.k >= 32768) {
    // persistent over ranges of chains, at most T * E of them (with fewer
    // chains than about 64 ranges, one chain per lane over many small
    // workgroups spreads them over more CUs); a range holds at most
    // 512 / k + 2 tokens, whose x rows a stage holds
    const long long ranges = ((long long)g.T * g.E + GATE_CHAIN_STAGED_W - 1) / GATE_CHAIN_STAGED_W;
    // two workgroups per CU (the kernel's registers and LDS allow it)
    const int grid = (int)std::min<long long>(ranges, 512);
    if (g.k >= 8) gate_chain_staged_kernel<72, 3><<<grid, GATE_CHAIN_STAGED_W, 0, s>>>(g);
    else gate_chain_staged_kernel<136, 2><<<grid, GATE_CHAIN_STAGED_W, 0, s>>>(g);
  } else {
    gate_chain_kernel<<<std::min(16384, std::max(1, (g.T * g.k * 3 / 2 + WAVE - 1) / WAVE)), WAVE, 0, s>>>(g);
  }
  {
    const dim3 grid((g.T + NTH - 1) / NTH);
    const TableArgs t = tab ? *tab : TableArgs{};
    auto final_ = [&](auto epl) {
      constexpr int EPL = decltype(epl)::value;
      if (tab) gate_final_kernel<EPL, true><<<grid, NTH, 0, s>>>(g, t);
      else gate_final_kernel<EPL, false><<<grid, NTH, 0, s>>>(g, t);
    };
    if (g.E <= 16) final_(std::integral_constant<int, 1>{});
    else if (g.E <= 32) final_(std::integral_constant<int, 2>{});
    else if (g.E <= 64) final_(std::integral_constant<int, 4>{});
    else if (g.E <= 128) final_(std::integral_constant<int, 8>{});
    else final_(std::integral_constant<int, 32>{});
  }
  HIP_TRY(hipGetLastError());
  return MOE_OK;
}

}  // namespace

struct moe_handle {
  moe_config cfg;
  int N = 0;
  int T = 0, xmax = 0, mt_max = 0, ctl_words = 0, nblk = 0, nseg = 0, nt0 = 0, nt1 = 0, nsplit = 1;
  size_t arows = 0, orows = 0;  // row capacities of A and of Hbuf / O (the padded row map)
  int qx = 0, qxs = 0;
  moe_calib calib{};
  DevCalib dcal{};
  moe_ws_layout lay{};
  size_t off_calib = 0, off_blk_cnt = 0, off_blk_off = 0, off_blk_bad = 0, off_rbnd = 0, off_ctl[2] = {0, 0};
  size_t off_part = 0;
  size_t off_gate = 0;  // the gate's scratch (gate_layout)
  size_t off_sched = 0;  // schedule images, one per K option (sched_build_kernel)
  uint32_t calib_gen = 1;  // bumped by every moe_set_calib (a stored plan of an older table is stale)
  char* ws = nullptr;
  size_t ws_bytes = 0;
  const int32_t* tables_from = nullptr;
  unsigned long long launch_seq = 0;
  long long timeout_ticks = 200000000LL;  // 2 s at 100 MHz
  int inject_stall = 0;
  uint32_t jitter_seed = 0;
  int jitter_max = 0;
  long long* trace = nullptr;
  int trace_cap = 0, trace_rec0 = 0;
  bool resident_ok = false;  // the megakernel's N workgroups fit the GPU at once
  bool stack_resident_ok = false;  // the same for the stacked megakernel
};

namespace {

// Row capacities of the padded row map (common.h): every (segment, chunk)
// is rounded up to a 32-row group, at most MAX_K chunks per segment; plus
// one row tile of slack.  A holds the routed rows, Hbuf and O also the
// shared experts' rows (rank 0's tokens).
size_t a_rows(const moe_config& c) {
  const long long T = (long long)c.n_src_ranks * c.tokens_per_rank;
  const long long xmax = T * std::min(c.top_k, c.n_local_experts);
  return (size_t)(xmax + (long long)c.n_local_experts * MAX_K * ROW_ALIGN + BM);
}
size_t out_rows(const moe_config& c) {
  return a_rows(c) + (size_t)c.n_shared_experts * ((size_t)c.tokens_per_rank + MAX_K * ROW_ALIGN);
}

moe_status validate_cfg(const moe_config* c) {
  if (!c) return fail(MOE_ERR_INVALID_ARG, "config is NULL");
  if (c->n_src_ranks < 1 || c->n_src_ranks > 64) return fail(MOE_ERR_INVALID_ARG, "n_src_ranks must be in [1, 64]");
  if (c->tokens_per_rank < 1) return fail(MOE_ERR_INVALID_ARG, "tokens_per_rank must be >= 1");
  long long T = (long long)c->n_src_ranks * c->tokens_per_rank;
  if (T > (1 << 22)) return fail(MOE_ERR_UNSUPPORTED, "T = %lld tokens exceeds 2^22", T);
  if (c->hidden < 64 || c->hidden % 64 || c->hidden > 16384)
    return fail(MOE_ERR_INVALID_ARG, "hidden must be a multiple of 64 in [64, 16384]");
  if (c->ffn < 64 || c->ffn % 64 || c->ffn > 32768)
    return fail(MOE_ERR_INVALID_ARG, "ffn must be a multiple of 64 in [64, 32768]");
  if (c->n_experts < 1 || c->n_experts > MAX_E) return fail(MOE_ERR_INVALID_ARG, "n_experts must be in [1, %d]", MAX_E);
  if (c->top_k < 1 || c->top_k > MAX_TOPK || c->top_k > c->n_experts)
    return fail(MOE_ERR_INVALID_ARG, "top_k must be in [1, min(E, %d)]", MAX_TOPK);
  if (c->n_local_experts < 1 || c->n_local_experts > MAX_EL)
    return fail(MOE_ERR_INVALID_ARG, "n_local_experts must be in [1, %d]", MAX_EL);
  if (c->first_local_expert < 0 || c->first_local_expert + c->n_local_experts > c->n_experts)
    return fail(MOE_ERR_INVALID_ARG, "local experts [e0, e0+E_l) must lie in [0, E)");
  if (c->n_shared_experts < 0 || c->n_shared_experts > MAX_S)
    return fail(MOE_ERR_INVALID_ARG, "n_shared_experts must be in [0, %d]", MAX_S);
  if (c->n_workers < 0) return fail(MOE_ERR_INVALID_ARG, "n_workers must be >= 0");
  if (c->gemm1_split != 0 && c->gemm1_split != 1 && c->gemm1_split != 2 && c->gemm1_split != 4 &&
      c->gemm1_split != 8)
    return fail(MOE_ERR_INVALID_ARG, "gemm1_split must be 0, 1, 2, 4 or 8");
  if (c->gemm1_split > 1 && c->ffn % (32 * c->gemm1_split))
    return fail(MOE_ERR_INVALID_ARG, "ffn must be a multiple of 32 * gemm1_split");
  const long long orows = (long long)out_rows(*c);
  if (orows > (1LL << 31) / 2) return fail(MOE_ERR_UNSUPPORTED, "too many routed rows");
  // dispatch addresses the row buffer A, the split reduction the output rows
  // O, with 32-bit byte offsets
  if (orows * (long long)c->hidden * 2 >= (1LL << 32))
    return fail(MOE_ERR_UNSUPPORTED, "routed rows (T * min(k, E_l) + S * T_r, padded) x H bf16 exceed 4 GiB");
  return MOE_OK;
}

moe_status validate_calib(const moe_calib* k, int N) {
  if (k->n_c < 1 || k->n_c > MOE_CALIB_MAX_C) return fail(MOE_ERR_INVALID_ARG, "calib n_c must be in [1, %d]", MOE_CALIB_MAX_C);
  if (k->n_k < 1 || k->n_k > MOE_CALIB_MAX_K) return fail(MOE_ERR_INVALID_ARG, "calib n_k must be in [1, %d]", MOE_CALIB_MAX_K);
  for (int i = 0; i < k->n_c; ++i) {
    if (k->c[i] < 1 || k->c[i] >= N) return fail(MOE_ERR_INVALID_ARG, "calib c[%d] = %d outside [1, N-1], N = %d", i, k->c[i], N);
    if (i && k->c[i] <= k->c[i - 1]) return fail(MOE_ERR_INVALID_ARG, "calib c must ascend");
    if (!(k->bw_bytes_per_s[i] > 0) || !(k->comp_flop_per_s[i] > 0) || !std::isfinite(k->bw_bytes_per_s[i]) ||
        !std::isfinite(k->comp_flop_per_s[i]))
      return fail(MOE_ERR_INVALID_ARG, "calib throughputs must be positive and finite");
  }
  for (int j = 0; j < k->n_k; ++j) {
    int K = k->k_chunks[j];
    if (K != 1 && K != 2 && K != 4 && K != 8) return fail(MOE_ERR_INVALID_ARG, "calib K must be 1, 2, 4 or 8");
    if (j && K <= k->k_chunks[j - 1]) return fail(MOE_ERR_INVALID_ARG, "calib K must ascend");
    if (!(k->eff_chunk[j] > 0) || k->eff_chunk[j] > 1) return fail(MOE_ERR_INVALID_ARG, "eff_chunk must be in (0, 1]");
  }
  if (!(k->alpha >= 0 && k->alpha <= 1)) return fail(MOE_ERR_INVALID_ARG, "alpha must be in [0, 1]");
  if (k->static_c < 1 || k->static_c >= N) return fail(MOE_ERR_INVALID_ARG, "static_c must be in [1, N-1]");
  if (!(k->bw_all_bytes_per_s >= 0) || !std::isfinite(k->bw_all_bytes_per_s))
    return fail(MOE_ERR_INVALID_ARG, "bw_all must be >= 0 and finite");
  if (k->steal_window != MOE_WINDOW_PLAIN && k->steal_window != MOE_WINDOW_MOVE_STEAL &&
      k->steal_window != MOE_WINDOW_LAST_COMBINE)
    return fail(MOE_ERR_INVALID_ARG, "steal_window must be a MOE_WINDOW_* value");
  if (k->steal_ceil != 0 && k->steal_ceil != 1) return fail(MOE_ERR_INVALID_ARG, "steal_ceil must be 0 or 1");
  return MOE_OK;
}

// Nominal MI355X curves used until a measured table is supplied.
void default_calib(int N, moe_calib* k) {
  memset(k, 0, sizeof *k);
  int n = 0;
  for (int c = 8; c <= 128 && c < N && n < MOE_CALIB_MAX_C; c += 8) {
    k->c[n] = c;
    k->bw_bytes_per_s[n] = std::min(40e9 * c, 5.0e12);
    k->comp_flop_per_s[n] = 4.0e12 * (N - c);
    ++n;
  }
  if (n == 0) {
    k->c[0] = std::max(1, N / 4);
    k->bw_bytes_per_s[0] = 40e9 * k->c[0];
    k->comp_flop_per_s[0] = 4.0e12 * (N - k->c[0]);
    n = 1;
  }
  k->n_c = n;
  k->n_k = 4;
  const int kk[4] = {1, 2, 4, 8};
  const double eff[4] = {1.0, 0.93, 0.85, 0.73};
  for (int j = 0; j < 4; ++j) { k->k_chunks[j] = kk[j]; k->eff_chunk[j] = eff[j]; }
  k->alpha = 0.5;
  k->literal_volumes = 0;
  int sc = (int)std::lround(N * 20.0 / 132.0 / 8.0) * 8;  // 20 of 132 SMs, rounded to XCD multiples
  k->static_c = std::min(std::max(sc, 1), N - 1);
  k->bw_all_bytes_per_s = 4.0e12;  // all workers copying together
  k->steal_window = MOE_WINDOW_MOVE_STEAL;
  k->steal_ceil = 1;
}

void to_dev(const moe_calib& k, DevCalib* d) {
  memset(d, 0, sizeof *d);
  d->n_c = k.n_c;
  for (int i = 0; i < k.n_c; ++i) { d->c[i] = k.c[i]; d->bw[i] = k.bw_bytes_per_s[i]; d->fl[i] = k.comp_flop_per_s[i]; }
  d->n_k = k.n_k;
  for (int j = 0; j < k.n_k; ++j) { d->kk[j] = k.k_chunks[j]; d->eff[j] = k.eff_chunk[j]; }
  d->alpha = k.alpha;
  d->literal = k.literal_volumes;
  d->static_c = k.static_c;
  d->bw_all = k.bw_all_bytes_per_s;
  d->steal_window = k.steal_window;
  d->steal_ceil = k.steal_ceil;
}

void compute_layout(moe_handle* h) {
  const moe_config& c = h->cfg;
  const int T = h->T, k = c.top_k, El = c.n_local_experts, R = c.n_src_ranks, S = c.n_shared_experts;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 256); return at; };
  moe_ws_layout& L = h->lay;
  L.slot = take(sizeof(int32_t) * (size_t)T * k);
  L.inv = take(sizeof(int32_t) * (size_t)std::max(h->xmax, 1));
  L.first_slot = take(sizeof(int32_t) * (size_t)T);
  L.off = take(sizeof(int32_t) * (size_t)(El + 1));
  L.sub_off = take(sizeof(int32_t) * (size_t)KOPT * El * SUBW);
  L.row_off = take(sizeof(int32_t) * (size_t)KOPT * (El + S) * SUBW);
  L.cnt_rank = take(sizeof(int32_t) * (size_t)El * R);
  L.uniq = take(sizeof(int32_t) * (size_t)R);
  L.stats = take(sizeof(int32_t) * ST_WORDS);
  L.plan = take(sizeof(moe_plan));
  L.err = take(sizeof(int32_t) * 4);
  h->off_calib = take(sizeof(DevCalib));
  h->off_gate = take(gate_layout(T, c.hidden, c.n_experts).total);
  h->off_sched = take(sizeof(int32_t) * (size_t)KOPT * SCHED_WORDS + sizeof(StoredPlan));
  h->off_blk_cnt = take(sizeof(int32_t) * (size_t)h->nblk * El);
  h->off_blk_off = take(sizeof(int32_t) * (size_t)h->nblk * El);
  h->off_blk_bad = take(sizeof(int32_t) * (size_t)h->nblk);
  h->off_rbnd = take(sizeof(int32_t) * (size_t)El * (R + 1));
  h->off_ctl[0] = take(sizeof(int32_t) * (size_t)h->ctl_words);
  h->off_ctl[1] = take(sizeof(int32_t) * (size_t)h->ctl_words);
  h->arows = a_rows(c);
  h->orows = out_rows(c);
  L.A = take(sizeof(uint16_t) * h->arows * c.hidden);
  L.Hbuf = take(sizeof(uint16_t) * h->orows * c.ffn);
  L.O = take(sizeof(uint16_t) * h->orows * c.hidden);
  // split-K partials of GEMM1: fp32 [split][row][H], rows as in O
  h->off_part = h->nsplit > 1 ? take(sizeof(float) * (size_t)h->nsplit * h->orows * c.hidden) : 0;
  L.total = o;
}

template <typename T>
T* at(moe_handle* h, size_t off) { return reinterpret_cast<T*>(h->ws + off); }

moe_status need_ws(moe_handle* h) {
  if (!h) return fail(MOE_ERR_INVALID_ARG, "handle is NULL");
  if (!h->ws) return fail(MOE_ERR_STATE, "no workspace bound (moe_set_workspace)");
  return MOE_OK;
}

TableArgs table_args(moe_handle* h, const int32_t* topk_idx) {
  TableArgs a{};
  a.topk_idx = topk_idx;
  a.slot = at<int32_t>(h, h->lay.slot);
  a.inv = at<int32_t>(h, h->lay.inv);
  a.first_slot = at<int32_t>(h, h->lay.first_slot);
  a.off = at<int32_t>(h, h->lay.off);
  a.sub_off = at<int32_t>(h, h->lay.sub_off);
  a.row_off = at<int32_t>(h, h->lay.row_off);
  a.cnt_rank = at<int32_t>(h, h->lay.cnt_rank);
  a.uniq = at<int32_t>(h, h->lay.uniq);
  a.stats = at<int32_t>(h, h->lay.stats);
  a.blk_cnt = at<int32_t>(h, h->off_blk_cnt);
  a.blk_off = at<int32_t>(h, h->off_blk_off);
  a.blk_bad = at<int32_t>(h, h->off_blk_bad);
  a.rbnd = at<int32_t>(h, h->off_rbnd);
  a.err = at<int32_t>(h, h->lay.err);
  a.T = h->T;
  a.Tr = h->cfg.tokens_per_rank;
  a.R = h->cfg.n_src_ranks;
  a.k = h->cfg.top_k;
  a.E = h->cfg.n_experts;
  a.e0 = h->cfg.first_local_expert;
  a.El = h->cfg.n_local_experts;
  a.nblk = h->nblk;
  a.S = h->cfg.n_shared_experts;
  a.tiles_per_row_tile = h->nt0 + h->nt1 * h->nsplit;
  return a;
}

}  // namespace


namespace {
// A persistent kernel's N workgroups wait on each other, so all of them must
// be resident at once (checked once per handle and kernel).
moe_status check_resident(moe_handle* h, const void* kernel, bool& ok) {
  if (ok) return MOE_OK;
  int dev = 0, cus = 0, per_cu = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  HIP_TRY(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, FNTH, 0));
  if ((long long)cus * per_cu < h->N)
    return fail(MOE_ERR_UNSUPPORTED, "n_workers = %d exceeds the %lld workgroups the GPU holds at once", h->N,
                (long long)cus * per_cu);
  ok = true;
  return MOE_OK;
}

FwdArgs fwd_args(moe_handle* h, const uint16_t* x, const int32_t* topk_idx, const float* topk_w, const void* packed,
                 uint16_t* y, int32_t mode, const moe_plan* forced) {
  const moe_config& c = h->cfg;
  const int cur = (int)(h->launch_seq & 1ULL);
  FwdArgs a{};
  a.T = h->T;
  a.Tr = c.tokens_per_rank;
  a.R = c.n_src_ranks;
  a.H = c.hidden;
  a.F = c.ffn;
  a.k = c.top_k;
  a.El = c.n_local_experts;
  a.S = c.n_shared_experts;
  a.e0 = c.first_local_expert;
  a.N = h->N;
  a.nt0 = h->nt0;
  a.nt1 = h->nt1;
  a.nsplit = h->nsplit;
  // movement units: as many as there are wavefronts on the workers (a whole
  // unit per wavefront while every worker still moves rows), at most DT / CT
  // tokens each
  {
    const int per = h->T / (h->N * (FNTH / WAVE));
    a.dt = per < 1 ? 1 : (per > DT ? DT : per);
    a.ct = per < 1 ? 1 : (per > CT ? CT : per);
  }
  a.xmax = h->xmax;
  a.mt_max = h->mt_max;
  a.ctl_words = h->ctl_words;
  a.qx = h->qx;
  a.qxs = h->qxs;
  a.x = x;
  a.topk_idx = topk_idx;
  a.topk_w = topk_w;
  a.w13 = static_cast<const uint16_t*>(packed);
  a.w2t = a.w13 ? a.w13 + (size_t)h->nseg * slab_rows(2 * c.ffn) * c.hidden : nullptr;
  a.y = y;
  a.slot = at<int32_t>(h, h->lay.slot);
  a.sub_off = at<int32_t>(h, h->lay.sub_off);
  a.row_off = at<int32_t>(h, h->lay.row_off);
  a.sched = at<int32_t>(h, h->off_sched);
  a.calib_gen = h->calib_gen;
  a.stats = at<int32_t>(h, h->lay.stats);
  a.A = at<uint16_t>(h, h->lay.A);
  a.Hb = at<uint16_t>(h, h->lay.Hbuf);
  a.O = at<uint16_t>(h, h->lay.O);
  a.part = h->nsplit > 1 ? at<float>(h, h->off_part) : nullptr;
  a.prow = h->orows;
  a.ctl = at<int32_t>(h, h->off_ctl[cur]);
  a.ctl_next = at<int32_t>(h, h->off_ctl[cur ^ 1]);
  a.err = at<int32_t>(h, h->lay.err);
  a.plan_out = at<moe_plan>(h, h->lay.plan);
  a.calib = at<DevCalib>(h, h->off_calib);
  a.mode = mode;
  a.move_steal = mode == MOE_MODE_DYNAMIC ? 1 : 0;
  a.forced = forced ? 1 : 0;
  if (forced) a.fplan = *forced;
  a.timeout_ticks = h->timeout_ticks;
  a.inject_stall = h->inject_stall;
  a.jitter_seed = h->jitter_seed;
  a.jitter_max = h->jitter_max;
  a.trace = h->trace;
  a.trace_cap = h->trace_cap;
  a.trace_rec0 = h->trace_rec0;
  a.serial_K = 1;
  a.static_disp = 1;
  return a;
}
}  // namespace

// ---- routing that allocates nothing ------------------------------------------
// The gate's scratch for moe_route_topk_static lives in this file-scope
// device array, so that the entry point needs no allocation.  Each GPU holds
// its own copy until the process ends.  Host code must not use the array's
// name as an address (it is a host-side stand-in): its device address is
// looked up once per device with that device current and kept in
// g_scratch_ptr, which is what the kernels receive.
static __device__ __align__(256) unsigned char scratch[MOE_ROUTE_STATIC_SCRATCH_BYTES];

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[SCRATCH_MAX_DEVICES] = {};

// the current device's address of `scratch` (looked up on its first use)
moe_status static_scratch(char** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES)
    return fail(MOE_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, SCRATCH_MAX_DEVICES);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(MOE_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return MOE_OK;
}
}  // namespace

extern "C" {

const char* moe_last_error(void) { return g_err.c_str(); }

moe_status moe_init(const moe_config* cfg, const moe_calib* calib, moe_handle** out) {
  if (!out) return fail(MOE_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  moe_status st = validate_cfg(cfg);
  if (st != MOE_OK) return st;
  int N = cfg->n_workers;
  if (N == 0) {
    int dev = 0, cus = 0;
    HIP_TRY(hipGetDevice(&dev));
    HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    N = cus;
  }
  if (N < 2) return fail(MOE_ERR_INVALID_ARG, "need at least 2 workers");
  moe_handle* h = new moe_handle();
  h->cfg = *cfg;
  h->N = N;
  h->T = cfg->n_src_ranks * cfg->tokens_per_rank;
  h->xmax = h->T * std::min(cfg->top_k, cfg->n_local_experts);
  h->nseg = cfg->n_local_experts + cfg->n_shared_experts;
  h->mt_max = (h->xmax + cfg->n_shared_experts * cfg->tokens_per_rank) / BM + MAX_K * h->nseg + 1;
  h->nblk = (h->T + NTH - 1) / NTH;
  h->nt0 = (2 * cfg->ffn + BN - 1) / BN;
  h->nt1 = (cfg->hidden + BN - 1) / BN;
  // split GEMM1 (K = F) when F is large against H, so its tiles are about as
  // long as GEMM0's (K = H) and there are enough of them to fill the CUs
  if (cfg->gemm1_split) {
    h->nsplit = cfg->gemm1_split;
  } else {
    h->nsplit = cfg->ffn >= 3 * cfg->hidden ? 4 : (2 * cfg->ffn >= 3 * cfg->hidden ? 2 : 1);
    while (h->nsplit > 1 && cfg->ffn % (32 * h->nsplit)) h->nsplit /= 2;
  }
  // readiness counters per row tile (dispatched rows, GEMM0 columns, GEMM1
  // columns) and, when GEMM1 is split, split arrivals per (row, column) tile
  h->ctl_words = CTL_READY + (3 * h->mt_max + (h->nsplit > 1 ? h->mt_max * h->nt1 : 0)) * CTL_PAD;
  // per (stage, slab class) tile queue heads of the megakernel, then of the
  // serial GEMM kernels
  h->qx = h->ctl_words;
  h->qxs = h->qx + 2 * MAX_K * NXCD * CTL_PAD;
  h->ctl_words = h->qxs + 2 * MAX_K * NXCD * CTL_PAD;
  if (calib) {
    st = validate_calib(calib, N);
    if (st != MOE_OK) { delete h; return st; }
    h->calib = *calib;
  } else {
    default_calib(N, &h->calib);
  }
  to_dev(h->calib, &h->dcal);
  compute_layout(h);
  *out = h;
  return MOE_OK;
}

moe_status moe_destroy(moe_handle* h) {
  delete h;
  return MOE_OK;
}

moe_status moe_set_calib(moe_handle* h, const moe_calib* calib) {
  if (!h || !calib) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  moe_status st = validate_calib(calib, h->N);
  if (st != MOE_OK) return st;
  h->calib = *calib;
  to_dev(h->calib, &h->dcal);
  h->calib_gen++;
  if (h->ws) HIP_TRY(hipMemcpy(h->ws + h->off_calib, &h->dcal, sizeof(DevCalib), hipMemcpyHostToDevice));
  return MOE_OK;
}

moe_status moe_get_calib(const moe_handle* h, moe_calib* out) {
  if (!h || !out) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  *out = h->calib;
  return MOE_OK;
}

moe_status moe_set_jitter(moe_handle* h, uint32_t seed, int32_t max_sleeps) {
  if (!h) return fail(MOE_ERR_INVALID_ARG, "handle is NULL");
  if (max_sleeps < 0 || max_sleeps > 4096) return fail(MOE_ERR_INVALID_ARG, "max_sleeps must be in [0, 4096]");
  h->jitter_seed = seed;
  h->jitter_max = max_sleeps;
  return MOE_OK;
}

moe_status moe_set_timeout_ms(moe_handle* h, double ms, int32_t inject_stall) {
  if (!h) return fail(MOE_ERR_INVALID_ARG, "handle is NULL");
  if (!(ms >= 0) || ms > 600000.0) return fail(MOE_ERR_INVALID_ARG, "timeout must be in [0, 600000] ms");
  h->timeout_ticks = (long long)(ms * 1e5);
  h->inject_stall = inject_stall ? 1 : 0;
  return MOE_OK;
}

moe_status moe_workspace_size(const moe_handle* h, size_t* bytes) {
  if (!h || !bytes) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  *bytes = h->lay.total;
  return MOE_OK;
}

moe_status moe_workspace_layout(const moe_handle* h, moe_ws_layout* out) {
  if (!h || !out) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  *out = h->lay;
  return MOE_OK;
}

moe_status moe_set_workspace(moe_handle* h, void* ws, size_t bytes, void* stream) {
  if (!h || !ws) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(MOE_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (bytes < h->lay.total) return fail(MOE_ERR_INVALID_ARG, "workspace too small: %zu < %zu", bytes, h->lay.total);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  h->ws = static_cast<char*>(ws);
  h->ws_bytes = bytes;
  h->tables_from = nullptr;
  h->launch_seq = 0;
  // control words: both counter sets, error word, stats, plan
  const size_t ctl_bytes = h->off_ctl[1] + sizeof(int32_t) * (size_t)h->ctl_words - h->lay.stats;
  zero_i32_kernel<<<256, NTH, 0, s>>>(at<int32_t>(h, h->lay.stats), (int)(ctl_bytes / 4));
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(h->ws + h->off_calib, &h->dcal, sizeof(DevCalib), hipMemcpyHostToDevice, s));
  HIP_TRY(hipStreamSynchronize(s));
  return MOE_OK;
}

moe_status moe_packed_weights_size(const moe_handle* h, size_t* bytes) {
  if (!h || !bytes) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  const long long H = h->cfg.hidden, F = h->cfg.ffn;
  *bytes = (size_t)h->nseg * (size_t)(slab_rows(2 * F) * H + slab_rows(H) * F) * sizeof(uint16_t);
  return MOE_OK;
}

moe_status moe_pack_weights(moe_handle* h, const uint16_t* w1, const uint16_t* w3, const uint16_t* w2,
                            const uint16_t* ws1, const uint16_t* ws3, const uint16_t* ws2, void* packed,
                            void* stream) {
  if (!h || !w1 || !w3 || !w2 || !packed) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  const int El = h->cfg.n_local_experts, S = h->cfg.n_shared_experts, H = h->cfg.hidden, F = h->cfg.ffn;
  if (S > 0 && (!ws1 || !ws3 || !ws2)) return fail(MOE_ERR_INVALID_ARG, "shared-expert weights are NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint16_t* w13 = static_cast<uint16_t*>(packed);
  uint16_t* w2t = w13 + (size_t)h->nseg * slab_rows(2 * F) * H;
  auto launch = [&](const uint16_t* src, uint16_t* dst, int nseg, int rows, int cols, long long stride,
                    int inter, int which) -> moe_status {
    if (nseg == 0) return MOE_OK;
    PackArgs a{src, dst, rows, cols, stride, inter, which};
    dim3 grid((cols + 31) / 32, (rows + 31) / 32, nseg);
    pack_transpose_kernel<<<grid, NTH, 0, s>>>(a);
    HIP_TRY(hipGetLastError());
    return MOE_OK;
  };
  const long long s13 = slab_rows(2 * F) * H, s2 = slab_rows(H) * F;
  moe_status st;
  auto pad = [&](uint16_t* dst, int R, int K, long long stride) -> moe_status {
    if (slab_rows(R) == R) return MOE_OK;
    PadArgs a{dst, h->nseg, R, K, stride};
    pack_pad_kernel<<<256, NTH, 0, s>>>(a);
    HIP_TRY(hipGetLastError());
    return MOE_OK;
  };
  if ((st = pad(w13, 2 * F, H, s13)) != MOE_OK) return st;
  if ((st = pad(w2t, H, F, s2)) != MOE_OK) return st;
  if ((st = launch(w1, w13, El, H, F, s13, 1, 0)) != MOE_OK) return st;
  if ((st = launch(w3, w13, El, H, F, s13, 1, 1)) != MOE_OK) return st;
  if ((st = launch(w2, w2t, El, F, H, s2, 0, 0)) != MOE_OK) return st;
  if (S > 0) {
    if ((st = launch(ws1, w13 + El * s13, S, H, F, s13, 1, 0)) != MOE_OK) return st;
    if ((st = launch(ws3, w13 + El * s13, S, H, F, s13, 1, 1)) != MOE_OK) return st;
    if ((st = launch(ws2, w2t + El * s2, S, F, H, s2, 0, 0)) != MOE_OK) return st;
  }
  return MOE_OK;
}

// The routing tables' kernels on `s`; counted: the counting step already ran
// (the routing's last kernel did it on the ids it chose).
static moe_status launch_tables(moe_handle* h, const int32_t* topk_idx, hipStream_t s, bool counted) {
  TableArgs a = table_args(h, topk_idx);
  if (!counted) tab_count_kernel<<<h->nblk, NTH, 0, s>>>(a);
  tab_scan_kernel<<<1, TAB_SCAN_THREADS, 0, s>>>(a);
  tab_perm_kernel<<<h->nblk, NTH, 0, s>>>(a);
  tab_finalize_kernel<<<1, NTH, 0, s>>>(a);
  // the launches' schedules for every chunk option, from these tables
  sched_build_kernel<<<KOPT, FNTH, 0, s>>>(fwd_args(h, nullptr, topk_idx, nullptr, nullptr, nullptr, MOE_MODE_DYNAMIC, nullptr));
  HIP_TRY(hipGetLastError());
  h->tables_from = topk_idx;
  return MOE_OK;
}

moe_status moe_build_tables(moe_handle* h, const int32_t* topk_idx, void* stream) {
  moe_status st = need_ws(h);
  if (st != MOE_OK) return st;
  if (!topk_idx) return fail(MOE_ERR_INVALID_ARG, "topk_idx is NULL");
  return launch_tables(h, topk_idx, reinterpret_cast<hipStream_t>(stream), false);
}

moe_status moe_route(moe_handle* h, const uint16_t* x, const uint16_t* wg, const float* logit_bias, int32_t top_k,
                     int32_t* topk_idx, float* topk_w, void* stream) {
  moe_status st = need_ws(h);
  if (st != MOE_OK) return st;
  if (!x || !wg || !topk_idx || !topk_w) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  if (top_k != h->cfg.top_k) return fail(MOE_ERR_INVALID_ARG, "top_k %d differs from the configured %d", top_k, h->cfg.top_k);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  GateArgs g{};
  g.x = x;
  g.wg = wg;
  g.bias = logit_bias;
  g.topk_idx = topk_idx;
  g.topk_w = topk_w;
  g.T = h->T;
  g.H = h->cfg.hidden;
  g.E = h->cfg.n_experts;
  g.k = top_k;
  // the chain counter goes to the layer's stats (word ST_CANDS, reported)
  bind_gate(g, h->ws + h->off_gate, gate_layout(g.T, g.H, g.E), at<int32_t>(h, h->lay.stats));
  const TableArgs ta = table_args(h, topk_idx);
  st = launch_gate(g, s, &ta);
  if (st != MOE_OK) return st;
  return launch_tables(h, topk_idx, s, true);
}

moe_status moe_set_trace(moe_handle* h, void* buf, int64_t bytes) {
  if (!h) return fail(MOE_ERR_INVALID_ARG, "handle is NULL");
  // header, one record count per wavefront of the launch (64-byte aligned),
  // then one segment of trace_cap records per wavefront
  const int64_t nseg = (int64_t)h->N * (FNTH / WAVE);
  const int64_t hdr = TRACE_HDR + (4 * nseg + 63) / 64 * 64;
  if (buf && bytes < hdr + 32 * nseg)
    return fail(MOE_ERR_INVALID_ARG, "trace buffer needs at least %lld bytes (one record per wavefront)",
                (long long)(hdr + 32 * nseg));
  h->trace = static_cast<long long*>(buf);
  h->trace_rec0 = (int)(hdr / 8);
  h->trace_cap = buf ? (int)std::min<int64_t>((bytes - hdr) / 32 / nseg, 1 << 20) : 0;
  return MOE_OK;
}

moe_status moe_forward(moe_handle* h, const uint16_t* x, const int32_t* topk_idx, const float* topk_w,
                       const void* packed, uint16_t* y, int32_t mode, const moe_plan* forced, void* stream) {
  moe_status st = need_ws(h);
  if (st != MOE_OK) return st;
  if (!x || !topk_idx || !topk_w || !packed || !y) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  if (mode != MOE_MODE_DYNAMIC && mode != MOE_MODE_STATIC && mode != MOE_MODE_SERIAL)
    return fail(MOE_ERR_INVALID_ARG, "unknown mode %d", mode);
  if (h->tables_from != topk_idx)
    return fail(MOE_ERR_STATE, "routing tables were not built from this topk_idx (call moe_route or moe_build_tables)");
  if (forced) {
    if (forced->c < 1 || forced->c >= h->N) return fail(MOE_ERR_INVALID_ARG, "forced c must be in [1, N-1]");
    if (forced->K != 1 && forced->K != 2 && forced->K != 4 && forced->K != 8)
      return fail(MOE_ERR_INVALID_ARG, "forced K must be 1, 2, 4 or 8");
    if (forced->n_steal < 0) return fail(MOE_ERR_INVALID_ARG, "forced n_steal must be >= 0");
    if (forced->final_all != 0 && forced->final_all != 1) return fail(MOE_ERR_INVALID_ARG, "forced final_all must be 0 or 1");
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FwdArgs a = fwd_args(h, x, topk_idx, topk_w, packed, y, mode, forced);
  if (mode == MOE_MODE_SERIAL) {
    serial_dispatch_kernel<<<h->N, FNTH, 0, s>>>(a);
    serial_gemm0_kernel<<<h->N, FNTH, 0, s>>>(a);
    serial_gemm1_kernel<<<h->N, FNTH, 0, s>>>(a);
    serial_combine_kernel<<<h->N, FNTH, 0, s>>>(a);
    HIP_TRY(hipGetLastError());
  } else {
    // a persistent kernel: its N workgroups wait on each other, so all of
    // them must be resident at once (checked once per handle).  It is an
    // ordinary launch: on an otherwise idle GPU one workgroup lands on each
    // CU; a cooperative launch would hold it until all earlier work on the
    // device has drained (~20 us a layer).
    st = check_resident(h, reinterpret_cast<const void*>(&moe_megakernel), h->resident_ok);
    if (st != MOE_OK) return st;
    moe_megakernel<<<h->N, FNTH, 0, s>>>(a);
    HIP_TRY(hipGetLastError());
  }
  h->launch_seq++;
  return MOE_OK;
}

moe_status moe_forward_stack(moe_handle* const* layers, int32_t n_layers, const uint16_t* x,
                             const int32_t* const* topk_idx, const float* const* topk_w, const void* const* packed,
                             uint16_t* const* y, int32_t mode, const moe_plan* forced, void* stream) {
  if (!layers || !x || !topk_idx || !topk_w || !packed || !y) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  if (n_layers < 1 || n_layers > MOE_STACK_MAX)
    return fail(MOE_ERR_INVALID_ARG, "n_layers must be in [1, %d]", MOE_STACK_MAX);
  if (mode != MOE_MODE_DYNAMIC && mode != MOE_MODE_STATIC)
    return fail(MOE_ERR_INVALID_ARG, "a stacked launch runs the megakernel modes only");
  if (forced) {
    if (forced->K != 1 && forced->K != 2 && forced->K != 4 && forced->K != 8)
      return fail(MOE_ERR_INVALID_ARG, "forced K must be 1, 2, 4 or 8");
    if (forced->n_steal < 0 || (forced->final_all != 0 && forced->final_all != 1))
      return fail(MOE_ERR_INVALID_ARG, "forced n_steal must be >= 0 and final_all 0 or 1");
  }
  const int N = layers[0] ? layers[0]->N : 0;
  for (int l = 0; l < n_layers; ++l) {
    moe_handle* h = layers[l];
    moe_status st = need_ws(h);
    if (st != MOE_OK) return st;
    if (h->N != N) return fail(MOE_ERR_INVALID_ARG, "layer %d has %d workers, layer 0 has %d", l, h->N, N);
    if (!topk_idx[l] || !topk_w[l] || !packed[l] || !y[l])
      return fail(MOE_ERR_INVALID_ARG, "NULL argument of layer %d", l);
    for (int m = 0; m < l; ++m)
      if (layers[m] == h) return fail(MOE_ERR_INVALID_ARG, "layer %d repeats the handle of layer %d", l, m);
    if (h->tables_from != topk_idx[l])
      return fail(MOE_ERR_STATE, "layer %d: routing tables were not built from its topk_idx", l);
    if (forced && (forced->c < 1 || forced->c >= N)) return fail(MOE_ERR_INVALID_ARG, "forced c must be in [1, N-1]");
  }
  moe_status st = check_resident(layers[0], reinterpret_cast<const void*>(&moe_megakernel_stack),
                                 layers[0]->stack_resident_ok);
  if (st != MOE_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  StackArgs sa{};
  sa.n = n_layers;
  for (int l = 0; l < n_layers; ++l) {
    FwdArgs& a = sa.layer[l];
    a = fwd_args(layers[l], x, topk_idx[l], topk_w[l], packed[l], y[l], mode, forced);
    // workers reach the later layers at different times: no dispatch unit
    // is owned by arrival ticket there; no timeline trace in a stacked launch
    a.static_disp = l == 0 ? 1 : 0;
    a.stack_next = l + 1 < n_layers ? 1 : 0;
    a.trace = nullptr;
  }
  moe_megakernel_stack<<<N, FNTH, 0, s>>>(sa);
  HIP_TRY(hipGetLastError());
  for (int l = 0; l < n_layers; ++l) layers[l]->launch_seq++;
  return MOE_OK;
}

moe_status moe_run_stages(moe_handle* h, const uint16_t* x, const int32_t* topk_idx, const float* topk_w,
                          const void* packed, uint16_t* y, int32_t stages, int32_t n_workers, int32_t K, void* stream) {
  moe_status st = need_ws(h);
  if (st != MOE_OK) return st;
  if (!x || !topk_idx || !topk_w || !packed || !y) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  if (stages <= 0 || stages > 15) return fail(MOE_ERR_INVALID_ARG, "stages must be a non-empty mask of bits 0..3");
  if (n_workers < 1 || n_workers > h->N) return fail(MOE_ERR_INVALID_ARG, "n_workers must be in [1, N]");
  if (K != 1 && K != 2 && K != 4 && K != 8) return fail(MOE_ERR_INVALID_ARG, "K must be 1, 2, 4 or 8");
  if (h->tables_from != topk_idx)
    return fail(MOE_ERR_STATE, "routing tables were not built from this topk_idx (call moe_route or moe_build_tables)");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FwdArgs a = fwd_args(h, x, topk_idx, topk_w, packed, y, MOE_MODE_SERIAL, nullptr);
  a.serial_K = K;
  // the first kernel clears the next control set; run it even when not asked
  // for, on zero tokens, so the control sets keep alternating
  if (stages & 1) {
    serial_dispatch_kernel<<<n_workers, FNTH, 0, s>>>(a);
  } else {
    FwdArgs z = a;
    z.T = 0;
    serial_dispatch_kernel<<<1, FNTH, 0, s>>>(z);
  }
  if (stages & 2) serial_gemm0_kernel<<<n_workers, FNTH, 0, s>>>(a);
  if (stages & 4) serial_gemm1_kernel<<<n_workers, FNTH, 0, s>>>(a);
  if (stages & 8) serial_combine_kernel<<<n_workers, FNTH, 0, s>>>(a);
  HIP_TRY(hipGetLastError());
  h->launch_seq++;
  return MOE_OK;
}

moe_status moe_get_plan(moe_handle* h, moe_plan* out, void* stream) {
  moe_status st = need_ws(h);
  if (st != MOE_OK) return st;
  if (!out) return fail(MOE_ERR_INVALID_ARG, "out is NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(hipMemcpyAsync(out, h->ws + h->lay.plan, sizeof(moe_plan), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return MOE_OK;
}

moe_status moe_sync_status(moe_handle* h, void* stream) {
  moe_status st = need_ws(h);
  if (st != MOE_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int32_t e = 0;
  HIP_TRY(hipStreamSynchronize(s));
  HIP_TRY(hipMemcpy(&e, h->ws + h->lay.err, sizeof e, hipMemcpyDeviceToHost));
  if (e) {
    zero_i32_kernel<<<1, 64, 0, s>>>(at<int32_t>(h, h->lay.err), 1);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipStreamSynchronize(s));
  }
  if (e & ERR_TIMEOUT) return fail(MOE_ERR_TIMEOUT, "a device-side wait timed out");
  if (e & ERR_ROUTING) return fail(MOE_ERR_ROUTING, "routing ids out of range or repeated within a row");
  return MOE_OK;
}

moe_status moe_plan_host(const moe_handle* h, double w_comp, double w_dispatch, double w_combine,
                         const int64_t* n_tiles, moe_plan* out) {
  if (!h || !n_tiles || !out) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  long long nt[MOE_CALIB_MAX_K];
  for (int j = 0; j < h->dcal.n_k; ++j) nt[j] = n_tiles[j];
  cost_model(h->dcal, h->N, w_comp, w_dispatch, w_combine, nt, out);
  return MOE_OK;
}

moe_status moe_tile_geometry(const moe_handle* h, int32_t* bm, int32_t* nt0, int32_t* nt1) {
  if (!h || !bm || !nt0 || !nt1) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  *bm = BM;
  *nt0 = h->nt0;
  *nt1 = h->nt1 * h->nsplit;
  return MOE_OK;
}

moe_status moe_route_topk_static(int32_t T, int32_t H, int32_t E, int32_t top_k, const uint16_t* x,
                                 const uint16_t* wg, const float* logit_bias, int32_t* topk_idx, float* topk_w,
                                 void* stream) {
  if (!x || !wg || !topk_idx || !topk_w) return fail(MOE_ERR_INVALID_ARG, "NULL argument");
  if (T < 1 || T > (1 << 22)) return fail(MOE_ERR_INVALID_ARG, "T = %d outside [1, 2^22]", T);
  if (H < 64 || H % 64 || H > 16384) return fail(MOE_ERR_INVALID_ARG, "H must be a multiple of 64 in [64, 16384]");
  if (E < 1 || E > MAX_E) return fail(MOE_ERR_INVALID_ARG, "E must be in [1, %d]", MAX_E);
  if (top_k < 1 || top_k > MAX_TOPK || top_k > E)
    return fail(MOE_ERR_INVALID_ARG, "top_k must be in [1, min(E, %d)]", MAX_TOPK);
  const GateLayout L = gate_layout(T, H, E);
  if (L.total > (size_t)MOE_ROUTE_STATIC_SCRATCH_BYTES)
    return fail(MOE_ERR_UNSUPPORTED, "T = %d, H = %d, E = %d needs %zu bytes of gate scratch, more than the %zu of "
                "the static scratch (use moe_route)", T, H, E, L.total, (size_t)MOE_ROUTE_STATIC_SCRATCH_BYTES);
  char* base = nullptr;
  moe_status st = static_scratch(&base);
  if (st != MOE_OK) return st;
  GateArgs g{};
  g.x = x;
  g.wg = wg;
  g.bias = logit_bias;
  g.topk_idx = topk_idx;
  g.topk_w = topk_w;
  g.T = T;
  g.H = H;
  g.E = E;
  g.k = top_k;
  // the chain counter (the one word that must start at zero) is cleared by
  // the first kernel of the gate; every other region is written before it
  // is read
  bind_gate(g, base, L, reinterpret_cast<int32_t*>(base + L.stats));
  return launch_gate(g, reinterpret_cast<hipStream_t>(stream), nullptr);
}

}  // extern "C"
