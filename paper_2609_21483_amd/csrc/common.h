// Device-side building blocks shared by the routing, forward and packing
// kernels of the MI355X (gfx950, CDNA4) MoE-layer library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/moe.h"

namespace moe {

// ---- fixed launch geometry ------------------------------------------------
constexpr int NTH = 256;        // threads per workgroup of the routing kernels
constexpr int FNTH = 512;       // threads per workgroup of the forward kernels (8 wave64s)
constexpr int WAVE = 64;

// grouped-GEMM tile: BM rows x BN columns (bf16 MFMA 32x32x16, see gemm.h)
constexpr int BM = 256;
constexpr int BN = 256;
constexpr int MAX_SPLIT = 8;    // split-K factor limit of GEMM1

// Packed expert weights are slab-tiled GEMM B operands: an [R][K] matrix
// (R output columns, K deep) is stored as ceil(R / 256) slabs of 256 rows;
// slab j holds its K / 32 k-steps one after the other, each a block of 256
// rows x 32 bf16 (row r of the block at r * 64 bytes).  Rows past R are zero.
constexpr int SLAB = 256;
constexpr int SLAB_K = 32;
__host__ __device__ inline long long slab_rows(long long R) { return (R + SLAB - 1) / SLAB * SLAB; }
// element offset of (row n, column k) in a slab-tiled [R][K] matrix
__host__ __device__ inline long long slab_index(long long n, long long k, long long K) {
  return ((n / SLAB) * (K / SLAB_K) + k / SLAB_K) * (SLAB * SLAB_K) + (n % SLAB) * SLAB_K + k % SLAB_K;
}

constexpr int DT = 8;           // most tokens per dispatch unit (one wavefront; DT * top_k <= 64)
constexpr int CT = 4;           // most tokens per combine unit (one wavefront)

constexpr int MAX_EL = 64;      // local experts
constexpr int MAX_S = 8;        // shared experts
constexpr int MAX_SEG = MAX_EL + MAX_S;
constexpr int MAX_K = 8;        // chunk count limit
constexpr int NLVL = 1;        // readiness levels of the routed row tiles of a stage
constexpr int MAX_TOPK = 8;
constexpr int MAX_E = 512;
constexpr int KOPT = 4;         // chunk options with stored offsets: K = 1, 2, 4, 8
constexpr int SUBW = 9;         // stored offsets per (K option, expert): K+1 <= 9

// Rows of A, Hbuf and O are grouped 32 to a group (the group-tiled operand
// layout of gemm.h: one 128-byte line holds two rows of a group).  Every
// (segment, chunk) starts on a group boundary, so no line holds rows of two
// segments or chunks: workers on different XCDs (each with its own L2) that
// wait for different readiness counters never share a line, and no L2 can
// cache a line of rows that are not written yet.  Row r of segment (seg, q)
// at chunk option K lies at row_off[kopt(K)][seg][q] + r; the padding rows
// at the end of a segment are never written nor read.
constexpr int ROW_ALIGN = 32;
__host__ __device__ inline int align_rows(int n) { return (n + ROW_ALIGN - 1) / ROW_ALIGN * ROW_ALIGN; }

__host__ __device__ inline int kopt_index(int K) { return K == 1 ? 0 : K == 2 ? 1 : K == 4 ? 2 : 3; }
__host__ __device__ inline int kopt_value(int i) { return 1 << i; }

// ---- control block: queue heads, readiness counters (int32 words) ------------
// Two sets are kept; launch n uses set n%2 and clears set (n+1)%2 for the next
// launch, so the layer is a single kernel launch with no host-side reset.
// Every counter has a 64-byte line of its own (CTL_PAD words), so pollers of
// one counter do not share a line with updates of another.
constexpr int CTL_PAD = 16;
constexpr int CTL_TICKET = 16;    // arrival ticket -> role
constexpr int CTL_ABORT = 32;     // set once any wait times out
constexpr int NSHARD = 64;        // movement-unit queue shards (one per lane of a wavefront)
constexpr int CTL_QC = 128;       // [NSHARD] combine-unit queue heads (CTL_PAD apart)
constexpr int NXCD = 8;           // XCDs of gfx950 (slab classes of the tile queues)
constexpr int CTL_QD = CTL_QC + NSHARD * CTL_PAD;     // [NSHARD] dispatch-unit queue heads
constexpr int CTL_READY = CTL_QD + NSHARD * CTL_PAD;  // [mt_max] dispatched rows per row tile (CTL_PAD apart),
// then [mt_max] GEMM0 column tiles finished per row tile (CTL_PAD apart),
// then [mt_max] GEMM1 (column tile, split) items finished per row tile (CTL_PAD apart)
static_assert(CTL_QC + NSHARD * CTL_PAD <= CTL_QD, "control block overlap");
static_assert(CTL_QD + NSHARD * CTL_PAD <= CTL_READY, "control block overlap");

// timeline trace buffer: header word 0 holds this tag (format of the layout below)
constexpr int TRACE_MAGIC = 0x31435254;  // "TRC1"
constexpr int TRACE_HDR = 64;            // header bytes; per-segment counts follow

// stats words written by the table builder
constexpr int ST_X = 0, ST_XLOCAL = 1, ST_XIN = 2, ST_ULOCAL = 3, ST_UIN = 4, ST_BADIDS = 5;
// written by the gate: candidates whose defined logit was evaluated (all tokens)
constexpr int ST_CANDS = 8;
// written by the table builder: GEMM tiles of the layer at each stored chunk
// option (KOPT words; the cost model's tile counts, Eq 14)
constexpr int ST_NTK = 10;
constexpr int ST_WORDS = 16;

// device error word values
constexpr int ERR_TIMEOUT = 1;
constexpr int ERR_ROUTING = 2;

// ---- bf16 -----------------------------------------------------------------
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN)
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
// two fp32 -> packed bf16 (lo in bits 0-15), round to nearest even, in one
// v_cvt_pk_bf16_f32; the same bits as f32_to_bf16 for every non-NaN value
typedef __bf16 bf16x2_hw_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_hw_t));
}

// ---- memory-model helpers (agent scope: every CU of every XCD) ---------------
__device__ __forceinline__ int ld_relaxed(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int fetch_add_relaxed(int* p, int v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_relaxed(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }  // 100 MHz

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

}  // namespace moe
