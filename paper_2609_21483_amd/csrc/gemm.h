// Grouped-GEMM tile for gfx950: C[256 x 256] = A[256 x K] * B[256 x K]^T on
// bf16 MFMA (v_mfma_f32_32x32x16_bf16, fp32 accumulation).
//
// A is either row-major (leading dimension lda) or group-tiled: 32-row
// groups, each 32-deep k-step of a group one 2 KiB block (32 rows x 64
// bytes), so a tile starting at any row reads whole lines too.  B, the packed
// expert weights, is slab-tiled: a slab of 256 rows stores each 32-deep k-step as one 16 KiB
// block (256 rows x 64 bytes), so a stage of B is one contiguous block and
// every DMA instruction covers eight whole 128-byte lines instead of sixteen
// half lines of 8 KiB-strided rows (measured at full chip: 10% less time per
// k-step of the mainloop).  Slabs are padded to 256 rows, so B is never read
// out of bounds.
//
// Workgroup of 8 wave64s (2 per SIMD), wave grid 2 (rows) x 4 (columns), each
// wave owns 128 x 64 outputs = 4 x 2 MFMA blocks (128 accumulator registers).
// The tile's eight 32-row blocks alternate between the two wave rows (wave
// row wm takes blocks wm, wm + 2, wm + 4, wm + 6), so a partly filled row
// tile spreads its valid rows over all four SIMDs.
// A and B stream through a 4-stage LDS ring of BK = 32 deep stages filled by
// direct global->LDS loads (global_load_lds_dwordx4), issued 3 stages ahead.
// Rows are 64 bytes; their 16-byte granules are XOR-swizzled by (row >> 1) & 3
// so fragment reads are free of bank conflicts.  The fragments of the second
// 16-deep slice of a stage are read while the MFMAs of the first run, and the
// next stage's barrier sits between the two slices.
//
// Ragged tiles: A rows past the valid count are loaded from the last valid
// row (never out of bounds); B columns past the matrix are the slab's padding
// rows.  Neither output is stored; every output element depends only on its
// own A row and B row.
#pragma once

#include "common.h"

namespace moe {

namespace gemm {

constexpr int TILE_M = 256, TILE_N = 256, KSTEP = 32, NSTAGE = 4;
constexpr int NWAVE = 8, WM = 2, WN = 4;
constexpr int TM = TILE_M / WM, TN = TILE_N / WN;   // 128 x 64 per wave
constexpr int MB = TM / 32, NB = TN / 32;           // 4 x 2 MFMA blocks
static_assert(MB == 4, "mainloop dispatches on 0..4 active row blocks");
constexpr int A_BYTES = TILE_M * KSTEP * 2, B_BYTES = TILE_N * KSTEP * 2;
constexpr int STAGE_BYTES = A_BYTES + B_BYTES;      // 32 KiB
constexpr int RING_BYTES = NSTAGE * STAGE_BYTES;    // 128 KiB
constexpr int A_INSTR = A_BYTES / 1024 / NWAVE;     // DMA instructions per wave per stage
constexpr int B_INSTR = B_BYTES / 1024 / NWAVE;
constexpr int INSTR = A_INSTR + B_INSTR;

typedef f32x16_t Acc[MB][NB];

__device__ __forceinline__ int swz(int row, int chunk) { return row * 4 + (chunk ^ ((row >> 1) & 3)); }

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// one 16-byte-per-lane DMA: M0 = wave's LDS destination, lane address =
// uniform base + 32-bit offset.  Issued through asm so that the waits stay
// under the mainloop's explicit control (the compiler would otherwise drain
// every outstanding DMA before each LDS read it cannot disambiguate).  No
// other code of these kernels keeps a value in M0 across this statement.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const char* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop

// values that are uniform by construction, made visibly uniform (SGPRs)
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const char*>(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// Uniform, opaque copy of a scalar: broadcast from the first lane (the value
// is uniform by construction) and hidden from the optimiser, so expressions
// built from it cannot be hoisted above this point.  Used on the scalars of
// each tile so that a persistent loop does not keep the address arithmetic of
// every epilogue live across the mainloop.
__device__ __forceinline__ int opaque(int v) {
  v = __builtin_amdgcn_readfirstlane(v);
  asm volatile("" : "+s"(v));
  return v;
}
__device__ __forceinline__ size_t opaque(size_t v) {
  uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  asm volatile("" : "+s"(lo), "+s"(hi));
  return ((size_t)hi << 32) | lo;
}
template <typename T>
__device__ __forceinline__ T* opaque(T* p) {
  return reinterpret_cast<T*>(opaque((size_t)p));
}

// Lane id through a volatile asm statement: values derived from it are
// recomputed where they are used instead of being hoisted out of a persistent
// loop and kept live (or spilled) across every mainloop.
__device__ __forceinline__ int lane_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

struct DmaOff {
  uint32_t a[A_INSTR], b[B_INSTR];
};

// A operand of a tile: row-major from its first row (gstride 0, lda
// elements per row), or group-tiled: `A` points at the group holding the
// tile's first row, which is row r0 (0..31) of that group, and consecutive
// groups are gstride bytes apart.
struct AOp {
  const uint16_t* p;
  int lda, r0, gstride, rows;
};
constexpr int GROUP = 32;                      // rows per group of a group-tiled operand
constexpr int GROUP_STEP = GROUP * KSTEP * 2;  // bytes per k-step block of a group

__device__ __forceinline__ void dma_offsets(DmaOff& o, const AOp& A) {
  const int lda = opaque(A.lda), a_rows = opaque(A.rows), r0 = opaque(A.r0), gs = opaque(A.gstride);
  const int lane = lane_here(), wave = opaque((int)(threadIdx.x >> 6));
#pragma unroll
  for (int i = 0; i < A_INSTR; ++i) {
    const int g = (wave * A_INSTR + i) * 64 + lane;
    const int row = g >> 2, c = (g & 3) ^ ((row >> 1) & 3);
    const int r = row < a_rows ? row : a_rows - 1;
    const int p = r0 + r;
    o.a[i] = gs ? (uint32_t)((p >> 5) * gs + (p & (GROUP - 1)) * (KSTEP * 2) + c * 16) : (uint32_t)(r * lda + c * 8) * 2u;
  }
#pragma unroll
  for (int i = 0; i < B_INSTR; ++i) {
    const int g = (wave * B_INSTR + i) * 64 + lane;
    const int row = g >> 2, c = (g & 3) ^ ((row >> 1) & 3);
    o.b[i] = (uint32_t)(row * (KSTEP * 2) + c * 16);
  }
}

// One k-step of A and B into a ring stage.  Every operand is a scalar
// computed once per tile (see mainloop), so the loop holds no vector
// register that was loaded from memory before it: a reload in front of the
// loop would otherwise make the compiler wait for every outstanding DMA at
// each iteration.
template <bool ADMA>
__device__ __forceinline__ void issue_stage(uint32_t lds_a, uint32_t lds_b, const char* Ak, const char* Bk,
                                            const DmaOff& o) {
  if constexpr (ADMA) {
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) dma16(Ak, o.a[i], lds_a + i * 1024);
  }
#pragma unroll
  for (int i = 0; i < B_INSTR; ++i) dma16(Bk, o.b[i], lds_b + i * 1024);
}

struct FragOff {
  uint32_t a[2], b[2];
};

__device__ __forceinline__ FragOff frag_offsets() {
  const int lane = lane_here(), wave = opaque((int)(threadIdx.x >> 6));
  const int wm = wave % WM, wn = wave / WM;
  const int ra = wm * 32 + (lane & 31), rb = wn * TN + (lane & 31);
  FragOff f;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int c = kk * 2 + (lane >> 5);
    f.a[kk] = (uint32_t)swz(ra, c) * 16u;
    f.b[kk] = (uint32_t)(A_BYTES + swz(rb, c) * 16);
  }
  return f;
}

// A wave's 32-row blocks are 64 rows (4096 bytes) apart and keep the same
// swizzle, so every fragment of a slice is a constant offset from the lane's
// base.  These load and multiply the first MBA blocks of the wave's rows (the
// blocks that hold valid rows of the tile; see mainloop).
template <int MBA>
__device__ __forceinline__ void load_frags(const char* stage, int kk, const FragOff& fo, bf16x8_t (&af)[MB],
                                           bf16x8_t (&bfr)[NB]) {
  if constexpr (MBA > 0) {
    const char* pa = stage + fo.a[kk];
    const char* pb = stage + fo.b[kk];
#pragma unroll
    for (int mb = 0; mb < MBA; ++mb) af[mb] = *reinterpret_cast<const bf16x8_t*>(pa + mb * (WM * 2048));
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bfr[nb] = *reinterpret_cast<const bf16x8_t*>(pb + nb * 2048);
  }
}

template <int MBA>
__device__ __forceinline__ void mfma_block(Acc& acc, const bf16x8_t (&af)[MB], const bf16x8_t (&bfr)[NB]) {
#pragma unroll
  for (int mb = 0; mb < MBA; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb], acc[mb][nb], 0, 0, 0);
}

// The mainloop of a wave that computes its first MBA 32-row blocks.  Wave w
// loads A's 32-row block w (its A_INSTR DMA instructions cover those rows)
// when ADMA, i.e. when the block holds a valid row; a block without one is
// neither loaded nor read (the waves that would multiply it skip it too), so
// a nearly empty row tile streams little more than its B operand.  Every
// instance passes the same barriers, so the waves of a workgroup may run
// different instances; the DMA waits count this wave's own instructions.
template <int MBA, bool ADMA>
__device__ __forceinline__ void mainloop_mb(Acc& acc, const AOp& A, const uint16_t* B, int Kd, char* ring) {
  constexpr int WI = ADMA ? INSTR : B_INSTR;  // DMA instructions of this wave per stage
  const int nk = Kd / KSTEP;
  DmaOff o;
  dma_offsets(o, A);
  const int a_step = opaque(A.gstride) ? GROUP_STEP : KSTEP * 2;  // bytes from one k-step of A to the next
  // scalars of the DMA issue: this wave's destinations in stage 0 and the
  // operand bases, pinned in scalar registers
  const int wave = opaque((int)(threadIdx.x >> 6));
  const uint32_t ring0 = (uint32_t)opaque((int)lds_u32(ring));
  const uint32_t la0 = ring0 + (uint32_t)(wave * A_INSTR * 1024);
  const uint32_t lb0 = ring0 + (uint32_t)(A_BYTES + wave * B_INSTR * 1024);
  const char* Ab = opaque(reinterpret_cast<const char*>(A.p));
  const char* Bb = opaque(reinterpret_cast<const char*>(B));
  auto st = [&](int s) { return ring + (s & (NSTAGE - 1)) * STAGE_BYTES; };
  auto issue = [&](int s) {
    const uint32_t so = (uint32_t)((s & (NSTAGE - 1)) * STAGE_BYTES);
    issue_stage<ADMA>(la0 + so, lb0 + so, Ab + (size_t)s * a_step, Bb + (size_t)s * B_BYTES, o);
  };
  issue(0);
  if (nk > 1) issue(1);
  if (nk > 2) issue(2);
  if (nk > 2) wait_vm<2 * WI>(); else if (nk > 1) wait_vm<WI>(); else wait_vm<0>();
  __builtin_amdgcn_s_barrier();
  compiler_fence();
  bf16x8_t fa0[MB], fb0[NB], fa1[MB], fb1[NB];
  const FragOff fo = frag_offsets();
  load_frags<MBA>(st(0), 0, fo, fa0, fb0);
  int s = 0;
  for (; s < nk - 3; ++s) {  // steady state: the stage 3 ahead is always issued
    load_frags<MBA>(st(s), 1, fo, fa1, fb1);
    mfma_block<MBA>(acc, fa0, fb0);
    wait_vm<WI>();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(s + 3);
    load_frags<MBA>(st(s + 1), 0, fo, fa0, fb0);
    mfma_block<MBA>(acc, fa1, fb1);
  }
  for (; s < nk; ++s) {  // drain
    load_frags<MBA>(st(s), 1, fo, fa1, fb1);
    mfma_block<MBA>(acc, fa0, fb0);
    if (s + 1 < nk) {
      if (s + 2 < nk) wait_vm<WI>(); else wait_vm<0>();
      __builtin_amdgcn_s_barrier();
      compiler_fence();
      load_frags<MBA>(st(s + 1), 0, fo, fa0, fb0);
    }
    mfma_block<MBA>(acc, fa1, fb1);
  }
  __builtin_amdgcn_s_barrier();
  compiler_fence();
}

// acc += A[0..A.rows) . B^T over k in [0, Kd); Kd % 32 == 0.  B points at
// the first k-step block of a 256-row slab of slab-tiled weights.
// ring: RING_BYTES of LDS.  Ends with a barrier (the ring may be reused).
// A wave computes only the 32-row blocks of its rows that hold valid rows
// (a_rows): the last row tile of an expert is often nearly empty, and its
// padding rows would otherwise cost as much MFMA work as valid ones.  Their
// accumulators stay zero and are never stored.
__device__ __forceinline__ void mainloop(Acc& acc, const AOp& A, const uint16_t* B, int Kd, char* ring) {
  const int wave = opaque((int)(threadIdx.x >> 6)), wm = wave % WM;
  const int rows = opaque(A.rows);
  const int left = rows - wm * 32;  // valid rows from the wave's first block on
  const int mba = left <= 0 ? 0 : min(MB, (left + WM * 32 - 1) / (WM * 32));
  static_assert(A_INSTR * 16 == 32, "wave w's A DMA covers 32-row block w");
  if (rows > wave * 32) {
    switch (mba) {
      case MB: mainloop_mb<MB, true>(acc, A, B, Kd, ring); break;
      case 3: mainloop_mb<3, true>(acc, A, B, Kd, ring); break;
      case 2: mainloop_mb<2, true>(acc, A, B, Kd, ring); break;
      case 1: mainloop_mb<1, true>(acc, A, B, Kd, ring); break;
      default: mainloop_mb<0, true>(acc, A, B, Kd, ring); break;
    }
  } else {
    switch (mba) {
      case MB: mainloop_mb<MB, false>(acc, A, B, Kd, ring); break;
      case 3: mainloop_mb<3, false>(acc, A, B, Kd, ring); break;
      case 2: mainloop_mb<2, false>(acc, A, B, Kd, ring); break;
      case 1: mainloop_mb<1, false>(acc, A, B, Kd, ring); break;
      default: mainloop_mb<0, false>(acc, A, B, Kd, ring); break;
    }
  }
}

__device__ __forceinline__ void zero(Acc& acc) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.0f;
}

// Output coordinates of accumulator element r of block (mb, nb): column
// col_l + nb*32 and row row_l + dr(mb, r) of the tile.
struct OutMap {
  int row_l, col_l;
};
__device__ __forceinline__ OutMap out_map(int cols_per_wave) {
  const int lane = lane_here(), wave = opaque((int)(threadIdx.x >> 6));
  const int wm = wave % WM, wn = wave / WM;
  return {wm * 32 + 4 * (lane >> 5), wn * cols_per_wave + (lane & 31)};
}
__device__ __forceinline__ int out_dr(int mb, int r) { return mb * (WM * 32) + 8 * (r >> 2) + (r & 3); }

// Epilogues write through 16- or 32-bit buffer stores.  With CP = SC1 the
// stores are agent-coherent: once they have completed (vmcnt 0) every XCD can
// read them, so the tile can be published without an L2 write-back.
constexpr int CP_PLAIN = 0, CP_SC1 = 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t out_rsrc(void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(uniform_ptr(static_cast<const char*>(p))), 0, -1,
                                           0x00020000);
}

// Epilogues, staged through LDS.  A lane holds one column of each 32 x 32
// accumulator block (out_map), so stores straight from the accumulators are
// 2-byte stores, 128 per lane for the 256 x 256 GEMM1 tile.  Instead each
// lane converts pairs of rows with one packed conversion, swaps the packed
// word with its neighbour (adjacent lanes hold adjacent columns) so that it
// holds two adjacent columns of one row, and writes 32-bit words into the
// free ring, row-major with a padded row stride (rows r and r + 4 of one
// write fall in different bank halves).  Then every thread stores whole
// 16-byte pieces of rows.  The barriers wait for LDS traffic only: the
// stores drain while the next tile starts.
constexpr int EPI_PAD = 16;  // bytes of padding per staged row

// Barrier for LDS traffic only: this wave's LDS operations have completed,
// then every wave meets.  (__syncthreads also waits for this wave's global
// stores, vmcnt(0): the whole write latency of the tile's output.)
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt((3 << 14) | (7 << 4) | 15);  // lgkmcnt(0); vmcnt, expcnt not waited for
  __builtin_amdgcn_s_barrier();
  compiler_fence();
}

__device__ __forceinline__ uint32_t swap_lane_pair(uint32_t v) {
  // quad_perm [1, 0, 3, 2]: lane l takes lane l ^ 1's value
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
}

// Stages accumulator pairs (rows r, r + 1 of a column) of the row blocks
// mb in [mb0, mb1) into `lds` as bf16 words of two adjacent columns, rows
// relative to row `row_off`.  vals(mb, j, r) gives the value of the lane's
// column j (0 .. ncol-1 per wave) at register r of block mb.
template <int NCOL, typename ValFn>
__device__ __forceinline__ void stage_pairs(char* lds, int stride, int mb0, int mb1, int row_off, int cols_per_wave,
                                            ValFn&& vals) {
  const int lane = lane_here(), wave = opaque((int)(threadIdx.x >> 6));
  const int wm = wave % WM, wn = wave / WM;
  const bool odd = lane & 1;
  const int col = wn * cols_per_wave + ((lane & 31) & ~1);
  const int rl = wm * 32 + 4 * (lane >> 5) + (odd ? 1 : 0) - row_off;
  // byte selector of v_perm_b32 over (q, p), bytes 0-3 from p and 4-7 from q:
  // an even lane keeps its low half and takes its neighbour's (row r),
  // an odd lane takes its neighbour's high half and keeps its own (row r + 1)
  const uint32_t sel = odd ? 0x03020706u : 0x05040100u;
  // unrolled over every block (the accumulators are registers); mb0 and mb1
  // are constants where the callers' loops are unrolled
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    if (mb < mb0 || mb >= mb1) continue;
#pragma unroll
    for (int j = 0; j < NCOL; ++j)
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const uint32_t p = pack_bf16x2(vals(mb, j, r), vals(mb, j, r + 1));
        const uint32_t q = swap_lane_pair(p);
        const uint32_t w = __builtin_amdgcn_perm(q, p, sel);
        const int row = rl + out_dr(mb, r);
        *reinterpret_cast<uint32_t*>(lds + row * stride + (col + j * 32) * 2) = w;
      }
  }
}

// GEMM0 epilogue through LDS into a group-tiled h (as store_silu_mul_tiled).
// ring: RING_BYTES of LDS, free (the mainloop ended with a barrier); ends
// with a barrier on the LDS traffic (the stores may still be in flight).
template <int CP>
__device__ __forceinline__ void store_silu_mul_tiled_lds(const Acc& acc, uint16_t* out, int r0, int gs, int out_rows,
                                                         int out_cols, char* ring) {
  constexpr int COLS = TN / 2 * WN;  // 128 h columns
  constexpr int STRIDE = COLS * 2 + EPI_PAD;
  static_assert(TILE_M * STRIDE <= RING_BYTES, "staged h tile fits the ring");
  r0 = opaque(r0);
  gs = opaque(gs);
  out_rows = opaque(out_rows);
  out_cols = opaque(out_cols);
  // SiLU(g) * u with the hardware reciprocal (about 1 ulp of fp32; the value
  // is rounded to bf16 next): the IEEE division's refinement sequence took 2
  // of the epilogue's 7 us per tile
  stage_pairs<1>(ring, STRIDE, 0, MB, 0, TN / 2, [&](int mb, int, int r) {
    const float g = acc[mb][0][r], u = acc[mb][1][r];
    return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
  });
  lds_barrier();
  const __amdgpu_buffer_rsrc_t rs = out_rsrc(out);
  constexpr int PPR = COLS / 8;  // 16-byte pieces per row
#pragma unroll
  for (int i = 0; i < TILE_M * PPR / (NWAVE * 64); ++i) {
    const int piece = (int)threadIdx.x + i * NWAVE * 64;
    const int row = piece / PPR, c = (piece % PPR) * 8;
    if (row < out_rows && c < out_cols) {
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(ring + row * STRIDE + c * 2);
      const int p = r0 + row;
      const uint32_t off = (uint32_t)((p >> 5) * gs + (c >> 5) * (GROUP * KSTEP) + (p & (GROUP - 1)) * KSTEP + (c & 31));
      __builtin_amdgcn_raw_buffer_store_b128(v, rs, off * 2u, 0, CP);
    }
  }
  lds_barrier();
}

// GEMM1 epilogue through LDS into a row-major O (as store_bf16), in two
// halves of 128 rows (a staged 256-row tile would exceed the ring).  Ends
// with a barrier on the LDS traffic (the stores may still be in flight).
template <int CP>
__device__ __forceinline__ void store_bf16_lds(const Acc& acc, uint16_t* out, int ldo, int out_rows, int out_cols,
                                               char* ring) {
  constexpr int COLS = TILE_N;
  constexpr int STRIDE = COLS * 2 + EPI_PAD;
  constexpr int HALF = TILE_M / 2;
  static_assert(HALF * STRIDE <= RING_BYTES, "staged half tile fits the ring");
  static_assert(MB % 2 == 0, "a half holds whole row blocks of every wave");
  ldo = opaque(ldo);
  out_rows = opaque(out_rows);
  out_cols = opaque(out_cols);
  const __amdgpu_buffer_rsrc_t rs = out_rsrc(out);
  constexpr int PPR = COLS / 8;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    stage_pairs<NB>(ring, STRIDE, h * MB / 2, (h + 1) * MB / 2, h * HALF, TN,
                    [&](int mb, int j, int r) { return acc[mb][j][r]; });
    lds_barrier();
#pragma unroll
    for (int i = 0; i < HALF * PPR / (NWAVE * 64); ++i) {
      const int piece = (int)threadIdx.x + i * NWAVE * 64;
      const int row = piece / PPR, c = (piece % PPR) * 8;
      if (h * HALF + row < out_rows && c < out_cols) {
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(ring + row * STRIDE + c * 2);
        const uint32_t off = (uint32_t)((h * HALF + row) * ldo + c);
        __builtin_amdgcn_raw_buffer_store_b128(v, rs, off * 2u, 0, CP);
      }
    }
    lds_barrier();
  }
}

// GEMM1 split-K epilogue: this split's fp32 partial into a row-major buffer
// (the combine adds the splits in a fixed order)
template <int CP>
__device__ __forceinline__ void store_f32(const Acc& acc, float* out, int ldo, int out_rows, int out_cols) {
  ldo = opaque(ldo);
  const __amdgpu_buffer_rsrc_t rs = out_rsrc(out);
  const OutMap m = out_map(TN);
  const uint32_t base = (uint32_t)(m.row_l * ldo + m.col_l);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int dr = out_dr(mb, r);
      if (m.row_l + dr < out_rows) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          if (m.col_l + nb * 32 < out_cols)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[mb][nb][r]), rs,
                                                  (base + (uint32_t)(dr * ldo) + nb * 32) * 4u, 0, CP);
      }
    }
}

}  // namespace gemm
}  // namespace moe
