// gfx950 kernels of libsplash_attn: split planner, paged MLA attend (whole
// histories, position shards, or listed top-k positions), LSE combine, page
// gather and device-data checks.  (The DOP regroup kernels are in dop.hip.)
//
// Attend kernel design (one persistent workgroup per compute unit):
//  * Work unit = (query row n with all H heads, page range).  Under a fold
//    plan each worker runs its own run of units; otherwise the planner's
//    queue (longest unit first) is dealt to the workers in a snake.  Neither
//    takes an atomic, so a worker knows its next unit ahead and issues that
//    unit's query and first steps before its current epilogue.
//  * 4 waves, one per SIMD.  For QK^T and the softmax wave w owns heads
//    [32w, 32w+32), whose query rows stay in VGPRs for the whole unit (36
//    16-byte MFMA B fragments); for PV it owns output columns [128w, +128)
//    of all heads, 256 accumulation registers per lane.
//  * KV is staged 32 rows (half a page, one "step") at a time straight from
//    HBM into LDS with 16-byte direct-to-LDS loads, through a ring of four
//    slots: step j (QK), step j-1 (PV) and two steps in flight (three slots
//    and one step in flight for bf16 top-k, whose resolved rows need the
//    room).  The dense variants read page ids from the block table through
//    the scalar cache.  The chunk order of each row is XOR-permuted by row so
//    the operand reads below spread over the LDS banks.
//  * Iteration j, behind one workgroup barrier: S^T[32 keys x 32 heads] =
//    K Q^T for step j as one chain of 36 v_mfma_f32_32x32x16_bf16 (K read
//    from LDS as the A operand), with the first PV MFMAs of step j-1 and the
//    loads of step j+2 spread through it; then the softmax of step j
//    interleaved with the remaining PV MFMAs of step j-1; then P of step j is
//    written to LDS for every wave's PV.  Steady-state iterations are
//    compiled without the checks for a unit's first and last steps.
//  * Softmax in base 2 against a reference fixed at the unit's first-step
//    max, so O is never rescaled in the loop; a logit more than 64 above the
//    reference makes the workgroup redo the unit from its true max (at most
//    two passes).  Numerator and denominator share the reference, so the
//    result is the same function.
//  * O^T[512 x heads] += V^T P^T on MFMA: P^T fragments come from the P
//    exchange area in LDS and V^T is read from the same staged rows with
//    ds_read_b64_tr_b16 (bf16) or ds_read_b64_tr_b8 (fp8) transposing loads.
//  * Epilogue: O/l goes through LDS so that every store writes whole rows;
//    an unsplit tile stores bf16 out and its LSE, a split unit an fp16
//    partial with a power-of-two scale per 128 columns and its LSE, which
//    merge_splits_kernel folds into the tile's result.
//  * fp8 cache: E4M3 codes convert exactly to bf16; the per-token scale is
//    applied in fp32 to the score and to P before P is rounded for PV.
//  * fp8 latent-row cache (656-byte rows: E4M3 latent with a power-of-two
//    scale per 128 columns, bf16 RoPE): K tiles convert with their scale;
//    for PV, wave w's output columns are tile w, so its P weights take the
//    keys' tile-w scales.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.hpp"
#include "splash_common.hpp"

namespace splash {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

#define LDS_AS __attribute__((address_space(3)))

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt[3:0], [15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier that does not drain outstanding global->LDS loads (a
// __syncthreads() would wait for every in-flight load).  LDS writes of this
// wave are completed first; the compiler may not move memory accesses across.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt((0x3F & 15) | (7 << 4) | (0 << 8) | ((0x3F >> 4) << 14));  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Opaque copy: keeps the compiler from hoisting work derived from v out of a loop.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

__device__ __forceinline__ unsigned pack_bf16x2(float a, float b) {
  bf16x2 v = __builtin_convertvector((f32x2){a, b}, bf16x2);
  return __builtin_bit_cast(unsigned, v);
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ unsigned pack_f16x2(float a, float b) {
  f16x2 v = __builtin_convertvector((f32x2){a, b}, f16x2);
  return __builtin_bit_cast(unsigned, v);
}

// Split partials are stored in fp16, each (slot, head) quarter of 128
// columns multiplied by 2^-e: e = 0 unless the quarter's largest magnitude
// m reaches 2^15, else e = floor(log2 m) - 14, so every stored value stays
// below 2^15 and rescales exactly.  The exponent of magnitude m is read from
// its bits (a zero m gives e = 0; e <= 114).
__device__ __forceinline__ uint32_t partial_exponent(float m) {
  const int32_t ex = (int32_t)((__builtin_bit_cast(uint32_t, m) >> 23) & 255u) - 127 - 14;
  return ex > 0 ? (uint32_t)ex : 0u;
}
// Four stored fp16 values (two dwords) back to fp32, times 2^e.
__device__ __forceinline__ f32x4 unpack_f16x4(uint32_t lo, uint32_t hi, int e) {
  const f32x2 a = __builtin_convertvector(__builtin_bit_cast(f16x2, lo), f32x2);
  const f32x2 b = __builtin_convertvector(__builtin_bit_cast(f16x2, hi), f32x2);
  return (f32x4){__builtin_amdgcn_ldexpf(a[0], e), __builtin_amdgcn_ldexpf(a[1], e), __builtin_amdgcn_ldexpf(b[0], e),
                 __builtin_amdgcn_ldexpf(b[1], e)};
}

// 8 E4M3 codes (two dwords) -> 8 bf16 (exact).
__device__ __forceinline__ bf16x8 fp8x8_to_bf16(u32x2 raw) {
  u32x4 r;
  r[0] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[0], 1.0f, false));
  r[1] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[0], 1.0f, true));
  r[2] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[1], 1.0f, false));
  r[3] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[1], 1.0f, true));
  return __builtin_bit_cast(bf16x8, r);
}

__device__ __forceinline__ float wave_xor32(float v) { return __shfl_xor(v, 32, 64); }

// ---- QK^T of the fp8 caches on the fp8 matrix pipe.  A bf16 query value
// has 8 significant bits and an E4M3 code 4, so after scaling a head's row
// by a power of two that puts its largest |q| in [128, 256), each value x is
// the sum of two codes: hi = rne(x), then lo = rne(x - hi), whose residual
// has at most 4 significant bits.  lo holds the residual times 2^4 and its
// MFMA scales it back by 2^-4 (the B operand's block scale), so the split is
// exact for |x| >= 2^-6 (2^-14 of the row's largest value); below that each
// term is off by at most 2^-14.  K enters as the cache's own codes (latent
// rows: with each tile's power-of-two scale as the A operand's block
// scale).  S = scale * (K hi^T + 2^-4 K lo^T), two 32x32x64 MFMAs per 64
// dims, with no per-step conversion of K.  The fp8 MFMA sums its products
// to about 2^-18 of their magnitude sum (measured), where the bf16 MFMA
// keeps fp32: a score is off by up to about 2^-18 * sum |q_i k_i| * scale.
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef short s16x2 __attribute__((ext_vector_type(2)));

// 32 bf16 values of one 64-dim block (16 dwords: values 0-15 in `a`, 16-31
// in `b`, two per dword, low half first) times `inv` -> hi codes into `a`,
// lo codes (residual times 2^4) into `b` (value v at byte v % 4 of dword
// v / 4).
__device__ __forceinline__ void split_query_block(i32x8& a, i32x8& b, float inv) {
  i32x8 hi, lo;
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    const uint32_t d0 = (uint32_t)(g < 4 ? a[2 * g] : b[2 * g - 8]);
    const uint32_t d1 = (uint32_t)(g < 4 ? a[2 * g + 1] : b[2 * g - 7]);
    const float x0 = __uint_as_float(d0 << 16) * inv, x1 = __uint_as_float(d0 & 0xFFFF0000u) * inv;
    const float x2 = __uint_as_float(d1 << 16) * inv, x3 = __uint_as_float(d1 & 0xFFFF0000u) * inv;
    s16x2 w = {0, 0};
    w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, x0, x1, 1.0f, false);
    w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, x2, x3, 1.0f, true);
    const int hw = __builtin_bit_cast(int, w);
    const f32x2 h01 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(hw, 1.0f, false);
    const f32x2 h23 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(hw, 1.0f, true);
    s16x2 v = {0, 0};
    v = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(v, (x0 - h01[0]) * 16.f, (x1 - h01[1]) * 16.f, 1.0f, false);
    v = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(v, (x2 - h23[0]) * 16.f, (x3 - h23[1]) * 16.f, 1.0f, true);
    hi[g] = hw;
    lo[g] = __builtin_bit_cast(int, v);
  }
  a = hi;
  b = lo;
}

// One 32x32x64 fp8 MFMA of the QK^T chain (VGPR accumulator, as mfma_qk)
// with E8M0 block scales: byte 0 of `ks` scales the lane's K block, byte 0
// of `qs` its query block, each by 2^(byte - 127).  K comes straight from
// LDS and the query codes were written at the unit's start; VALU_SRC adds
// the wait states a scale written by the VALU just before needs (the
// constant scales are opaque values made once, never rematerialised here).
template <bool FIRST, bool VALU_SRC>
__device__ __forceinline__ void mfma_qk8(f32x16& acc, const i32x8& k, const i32x8& q, int ks, int qs) {
  if constexpr (FIRST) {
    if constexpr (VALU_SRC)
      asm volatile("s_nop 2\n\tv_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, 0, %3, %4 op_sel_hi:[0,0,0]"
                   : "=v"(acc) : "v"(k), "v"(q), "v"(ks), "v"(qs));
    else
      asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, 0, %3, %4 op_sel_hi:[0,0,0]"
                   : "=v"(acc) : "v"(k), "v"(q), "v"(ks), "v"(qs));
  } else {
    if constexpr (VALU_SRC)
      asm volatile("s_nop 2\n\tv_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, %0, %3, %4 op_sel_hi:[0,0,0]"
                   : "+v"(acc) : "v"(k), "v"(q), "v"(ks), "v"(qs));
    else
      asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, %0, %3, %4 op_sel_hi:[0,0,0]"
                   : "+v"(acc) : "v"(k), "v"(q), "v"(ks), "v"(qs));
  }
}

// ============================================================== planner ===

// Pages of tile t: its whole causal prefix, or under a shard its keys in
// [key_begin[b], min(prefix, key_end[b])) (key_begin a page boundary), or
// for the top-k variant its list entries in groups of 64.
__device__ __forceinline__ int32_t dev_tile_pages(const int32_t* seq_lens, int32_t q_chunk, int32_t t,
                                                  const int32_t* key_begin, const int32_t* key_end,
                                                  const int32_t* topk_count) {
  if (topk_count) return ceil_div(topk_count[t], kPage);
  int32_t b = t / q_chunk, i = t - b * q_chunk;
  int32_t L = tile_keys(seq_lens[b], q_chunk, i);
  if (key_end) {
    const int32_t hi = min(L, key_end[b]), lo = key_begin[b];
    return hi > lo ? ceil_div(hi, kPage) - lo / kPage : 0;
  }
  return L > 0 ? ceil_div(L, kPage) : 0;
}

// Whole-wave reductions of the device library (DPP based, no LDS round trips).
extern "C" __device__ __attribute__((const)) long long __ockl_wfred_add_i64(long long);
extern "C" __device__ __attribute__((const)) long long __ockl_wfred_min_i64(long long);
extern "C" __device__ __attribute__((const)) float __ockl_wfred_max_f32(float);
extern "C" __device__ __attribute__((const)) float __ockl_wfred_add_f32(float);

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
template <typename T>
__device__ __forceinline__ T wave_max(T v) {
  for (int o = 32; o > 0; o >>= 1) {
    T w = __shfl_xor(v, o, 64);
    v = w > v ? w : v;
  }
  return v;
}

// Inclusive scan of one int per lane over the wave with DPP moves: prefix
// sums inside each row of 16 lanes (shifts 1, 2, 4, 8), then the row totals
// are broadcast into the following rows.
__device__ __forceinline__ int32_t wave_incl_scan(int32_t x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 -> rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 -> rows 2, 3
  return x;
}

// Inclusive running max of one non-negative int per lane over the wave (the
// same DPP pattern as the scan, with max for the add).
__device__ __forceinline__ int32_t wave_incl_max(int32_t x) {
  x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false));  // row_shr:1
  x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false));  // row_shr:2
  x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false));  // row_shr:4
  x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false));  // row_shr:8
  x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false));  // row_bcast:15 -> rows 1, 3
  x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false));  // row_bcast:31 -> rows 2, 3
  return x;
}

// Exclusive block scan of one int per thread (1024 threads); returns the
// exclusive prefix and writes the block total to *total.
__device__ int32_t block_exclusive_scan(int32_t v, int32_t* wave_buf, int32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t inc = wave_incl_scan(v);
  if (lane == 63) wave_buf[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    const int32_t x = lane < 16 ? wave_buf[lane] : 0;
    const int32_t run = wave_incl_scan(x);
    if (lane < 16) wave_buf[lane] = run - x;
    if (lane == 15) wave_buf[16] = run;
  }
  __syncthreads();
  int32_t res = wave_buf[wave] + inc - v;
  *total = wave_buf[16];
  __syncthreads();
  return res;
}

// Three exclusive block scans at once (one set of barriers for the three).
__device__ void block_exclusive_scan3(int32_t a, int32_t b, int32_t c, int32_t* wave_buf, int32_t* ea, int32_t* eb,
                                      int32_t* ec, int32_t* ta, int32_t* tb, int32_t* tc) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t ia = wave_incl_scan(a), ib = wave_incl_scan(b), ic = wave_incl_scan(c);
  if (lane == 63) {
    wave_buf[wave] = ia;
    wave_buf[17 + wave] = ib;
    wave_buf[34 + wave] = ic;
  }
  __syncthreads();
  if (wave == 0) {
    const int32_t xa = lane < 16 ? wave_buf[lane] : 0, xb = lane < 16 ? wave_buf[17 + lane] : 0,
                  xc = lane < 16 ? wave_buf[34 + lane] : 0;
    const int32_t ra = wave_incl_scan(xa), rb = wave_incl_scan(xb), rc = wave_incl_scan(xc);
    if (lane < 16) {
      wave_buf[lane] = ra - xa;
      wave_buf[17 + lane] = rb - xb;
      wave_buf[34 + lane] = rc - xc;
    }
    if (lane == 15) {
      wave_buf[16] = ra;
      wave_buf[33] = rb;
      wave_buf[50] = rc;
    }
  }
  __syncthreads();
  *ea = wave_buf[wave] + ia - a;
  *eb = wave_buf[17 + wave] + ib - b;
  *ec = wave_buf[34 + wave] + ic - c;
  *ta = wave_buf[16];
  *tb = wave_buf[33];
  *tc = wave_buf[50];
  __syncthreads();
}

__global__ __launch_bounds__(1024) void plan_kernel(PlanLaunch p) {
  __shared__ int32_t s_pages[kPlanLdsTiles];
  __shared__ int32_t s_ufirst[kPlanLdsTiles + 1];  // first unit of each tile (cached case)
  __shared__ int32_t s_sfirst[kPlanLdsTiles];      // first partial slot of each tile (cached case)
  __shared__ int64_t s_w[16][kNumCandidates + 1], s_s[16][kNumCandidates + 1];  // units, split units per tile slice
  __shared__ int32_t s_lhist[kMaxUnitPages + 1];  // units per length
  __shared__ int32_t s_lbase[kMaxUnitPages + 1];  // next queue slot per length
  __shared__ int32_t s_q[kMaxWorkers];            // fold plan: pages of each rank (0 past the last tile)
  __shared__ int32_t s_rt[kMaxWorkers];           // fold plan: tile of each rank
  __shared__ int32_t s_pm[kMaxWorkers / 2];       // fold plan: running max of the pair loads
  __shared__ int64_t s_red64[16];
  __shared__ int32_t s_red32[16];
  __shared__ int64_t s_cost[kNumCandidates + 1];
  __shared__ int32_t s_list[kNumCandidates + 1];  // candidate index of each distinct size
  __shared__ int32_t s_nd;                        // number of distinct sizes
  __shared__ UDiv s_udiv[kNumCandidates + 1];      // their division magic
  __shared__ int32_t s_cand[kNumCandidates + 1];
  __shared__ int32_t s_parts[kNumCandidates];  // parts of each candidate
  __shared__ int32_t s_scan[51];
  __shared__ int32_t s_chunk;
  __shared__ int64_t s_best;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t T = p.B * p.q_chunk;
  const bool cached = T <= kPlanLdsTiles;
  // A shard's result is always a partial: every unit writes a partial slot
  // (the combine turns each tile's parts into its fp32 result), and tiles
  // with no key in the shard are listed for the combine with no parts.
  const bool shard = p.key_end != nullptr;
  // tiles with no key (a shard's, or a top-k row with an empty list) are
  // listed for the combine with no parts, which writes out = 0, lse = -inf
  const bool list_empty = shard || p.topk_count != nullptr;
  int32_t* hdr = p.ws.header;
  auto pages_of = [&](int32_t t) -> int32_t {
    return cached ? s_pages[t] : dev_tile_pages(p.seq_lens, p.q_chunk, t, p.key_begin, p.key_end, p.topk_count);
  };

  // 1. page counts (cached), total and largest tile.
  int64_t tot = 0;
  int32_t mx = 0;
  for (int32_t t = tid; t < T; t += 1024) {
    const int32_t P = dev_tile_pages(p.seq_lens, p.q_chunk, t, p.key_begin, p.key_end, p.topk_count);
    if (cached) s_pages[t] = P;
    tot += P;
    mx = P > mx ? P : mx;
  }
  // the candidates' part counts: k + 1 for k < 64, then the geometric
  // recurrence of plan_candidate_parts (uniform, unrolled; lane i of wave 1
  // keeps step i)
  static_assert(kNumCandidates >= 64 && kNumCandidates - 64 <= 64, "candidate layout");
  if (wave == 0) s_parts[lane] = lane + 1;
  if (wave == 1) {
    int32_t parts = 64, mine = 0;
#pragma unroll
    for (int i = 0; i < kNumCandidates - 64; ++i) {
      parts += parts / 8;
      if (lane == i) mine = parts;
    }
    if (lane < kNumCandidates - 64) s_parts[64 + lane] = mine;
  }
  tot = __ockl_wfred_add_i64(tot);
  mx = __ockl_wfred_max_i32(mx);
  if (lane == 0) { s_red64[wave] = tot; s_red32[wave] = mx; }
  __syncthreads();
  tot = 0; mx = 0;
  for (int w = 0; w < 16; ++w) { tot += s_red64[w]; mx = s_red32[w] > mx ? s_red32[w] : mx; }
  const int64_t total_pages = tot;
  const int32_t max_pages = mx > 0 ? mx : 1;

  // 2. unit size: evaluate every candidate (and a forced size), take the argmin.
  // Wave 0 lists the distinct candidate sizes (a size equal to the previous
  // candidate's is left out: the argmin keeps the smaller index on ties
  // anyway).  Then every wave counts units and split units of listed
  // candidates over a slice of the tiles: with at most 64 sizes lane j of
  // wave w takes size j over the tiles t = w + 16i, otherwise sizes
  // 64 (w >> 3) + j over t = (w & 7) + 8i.  The slices meet in LDS; wave 0
  // adds them up, prices every size (one lane each) and takes the argmin.
  if (wave == 0) {
    int32_t nd = 0;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int k = 64 * r + lane;
      int32_t ck = 0;
      if (k < kNumCandidates) {
        ck = plan_candidate_size(s_parts[k], max_pages, p.unit_cap);
        if (k > 0 && plan_candidate_size(s_parts[k - 1], max_pages, p.unit_cap) == ck) ck = 0;
      } else if (k == kNumCandidates && p.forced_chunk > 0) {
        ck = p.forced_chunk < p.unit_cap ? p.forced_chunk : p.unit_cap;
      }
      if (k <= kNumCandidates) s_cand[k] = ck;
      const uint64_t keep = __builtin_amdgcn_ballot_w64(ck > 0);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(keep >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)keep, 0));
      if (ck > 0) {
        s_list[nd + below] = k;
        s_udiv[nd + below] = udiv_make((uint32_t)ck);  // once per size
      }
      nd += __builtin_popcountll(keep);
    }
    if (lane == 0) {
      s_nd = nd;
      s_cost[kNumCandidates] = INT64_MAX;
    }
  }
  __syncthreads();
  const int nd = s_nd;
  const bool wide = nd > 64;
  const int nsl = wide ? 8 : 16;  // tile slices
  {
    // With at most 32 sizes, 64 / np2 lanes share a size (np2: nd rounded up
    // to a power of two), each taking every (64 / np2)-th tile of the slice;
    // their sums meet by shuffles.  (uniform per wave)
    const int np2 = wide ? 64 : (nd <= 1 ? 1 : 1 << (32 - __builtin_clz((unsigned)(nd - 1))));
    const int sub = 64 / np2;
    const int j = wide ? 64 * (wave >> 3) + lane : (lane & (np2 - 1));
    const int part = wide ? 0 : lane / np2;
    const int slice = wide ? (wave & 7) : wave;
    int64_t W = 0, S = 0;
    if (j < nd) {
      const int32_t ck = s_cand[s_list[j]];
      const UDiv ud = s_udiv[j];
      auto count = [&](int32_t P) {
        const int32_t n = (int32_t)udiv((uint32_t)(P + ck - 1), ud);  // ceil(P / c)
        W += n;
        S += (n > 1 || shard) ? n : 0;
      };
      if (cached) {
#pragma unroll 4
        for (int32_t t = slice + nsl * part; t < T; t += nsl * sub) count(s_pages[t]);
      } else {
        for (int32_t t = slice + nsl * part; t < T; t += nsl * sub)
          count(dev_tile_pages(p.seq_lens, p.q_chunk, t, p.key_begin, p.key_end, p.topk_count));
      }
    }
    for (int off = np2; off < 64; off <<= 1) {
      W += __shfl_xor(W, off, 64);
      S += __shfl_xor(S, off, 64);
    }
    if (j < nd && part == 0) {
      s_w[slice][j] = W;
      s_s[slice][j] = S;
    }
  }
  __syncthreads();
  if (wave == 0) {
    // price every listed size (lane j, then j + 64), then the first minimum
    // (smallest candidate index on ties): the key puts the cost above the
    // candidate index (costs stay far below 2^56)
    int64_t best = INT64_MAX;
    for (int j = lane; j < nd; j += 64) {
      const int k = s_list[j];
      const int32_t ck = s_cand[k];
      int64_t W = 0, S = 0;
      for (int sl = 0; sl < nsl; ++sl) {
        W += s_w[sl][j];
        S += s_s[sl][j];
      }
      const bool ok = S <= p.ws.max_partials && W <= p.ws.max_units;
      const int64_t cost = ok ? plan_cost(ck, W, S, total_pages, max_pages, p.G, kPlanCosts) : INT64_MAX;
      if (k == kNumCandidates) s_cost[kNumCandidates] = cost;
      const int64_t key = (cost == INT64_MAX || k == kNumCandidates) ? INT64_MAX : ((cost << 7) | k);
      best = key < best ? key : best;
    }
    best = __ockl_wfred_min_i64(best);
    int bk = best == INT64_MAX ? kNumCandidates : (int)(best & 127);
    if (lane == 0) {
      if (bk >= kNumCandidates) bk = 0;
      s_best = best == INT64_MAX ? INT64_MAX : (best >> 7);
      if (p.forced_chunk > 0 && s_cost[kNumCandidates] != INT64_MAX) bk = kNumCandidates;
      s_chunk = s_cand[bk];
    }
  }
  __syncthreads();
  const int32_t c = s_chunk;

  // 2b. the fold plan (at most one tile per worker, no forced size): rank
  // the tiles by pages, then price every cap (thread C - 1 takes cap C) and
  // keep the cheapest; taken when it beats every unit size.  The busiest worker under cap C is
  // max(16 C + U, max_{j < nl(C)} v_j - 16 C) with v_j = 16 (q_j + q_{G-1-j})
  // + U + U [q_{G-1-j} > 0] independent of C, so a running max of v over j
  // and a binary search for nl(C) = #{r : q_r > C} price a cap in O(log G).
  bool fold = p.forced_chunk == 0 && !shard &&
              fold_applicable(T, p.G, kMaxWorkers, max_pages, total_pages, s_best, kPlanCosts, p.unit_cap);
  int32_t cap = 0, nl = 0;
  if (fold) {
    // counting sort of the tiles by pages, longest first: the histogram, the
    // number of tiles with more pages (thread i takes pages kMaxUnitPages -
    // i), then one atomic per tile (tiles of equal pages in whatever order
    // the atomics give; it decides only which worker runs which of them)
    for (int32_t i = tid; i <= kMaxUnitPages; i += 1024) s_lhist[i] = 0;
    __syncthreads();
    if (tid < T) atomicAdd(&s_lhist[s_pages[tid]], 1);  // 0 <= pages <= kMaxUnitPages
    __syncthreads();
    int32_t longer;
    s_lbase[kMaxUnitPages - tid] = block_exclusive_scan(s_lhist[kMaxUnitPages - tid], s_scan, &longer);
    if (tid == 0) s_lbase[0] = longer;  // empty tiles last
    __syncthreads();
    if (tid < T) {
      const int32_t P = s_pages[tid], r = atomicAdd(&s_lbase[P], 1);
      s_q[r] = P;
      s_rt[r] = tid;
    } else if (tid < p.G) {
      s_q[tid] = 0;
    }
    __syncthreads();
    const int32_t U = kPlanCosts.unit_x16, half = p.G / 2;
    int32_t v = 0;
    if (tid < half) {
      const int32_t qk = s_q[p.G - 1 - tid];
      v = 16 * (s_q[tid] + qk) + U + (qk > 0 ? U : 0);
    }
    v = wave_incl_max(v);  // running max inside the wave, then over the waves before
    if (lane == 63) s_red32[wave] = v;
    __syncthreads();
    for (int w = 0; w < wave; ++w) v = s_red32[w] > v ? s_red32[w] : v;
    if (tid < half) s_pm[tid] = v;
    __syncthreads();
    auto count_long = [&](int32_t C) {  // first rank with q_r <= C (q descends)
      int32_t lo = 0, hi = T;
      while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (s_q[mid] > C) lo = mid + 1; else hi = mid;
      }
      return lo;
    };
    const int32_t C = tid + 1;
    int64_t key = INT64_MAX;
    if (C < s_q[0]) {
      const int32_t n = count_long(C);
      if (2 * n <= p.G && 2 * n <= p.ws.max_partials) {
        int64_t mk = 16 * (int64_t)C + U;
        if (n > 0 && (int64_t)s_pm[n - 1] - 16 * C > mk) mk = (int64_t)s_pm[n - 1] - 16 * C;
        const int64_t cost = (int64_t)p.G * (mk + kPlanCosts.split_x16) + 2 * (int64_t)n * kPlanCosts.combine_x16;
        key = (cost << 10) | (kMaxUnitPages - C);  // ties: the larger cap
      }
    }
    key = __ockl_wfred_min_i64(key);
    __syncthreads();  // every wave is past its reads of s_red32
    if (lane == 0) s_red64[wave] = key;
    __syncthreads();
    key = INT64_MAX;
    for (int w = 0; w < 16; ++w) key = s_red64[w] < key ? s_red64[w] : key;
    fold = key != INT64_MAX && (key >> 10) < s_best;
    if (fold) {
      cap = kMaxUnitPages - (int32_t)(key & 1023);
      nl = count_long(cap);
    }
  }
  auto tile_units = [&](int32_t t, int32_t P, int32_t* n, int32_t* sp) {
    if (fold) {
      *n = P > cap ? 2 : (P > 0 ? 1 : 0);
      *sp = P > cap ? 2 : 0;
    } else {
      *n = P > 0 ? ceil_div(P, c) : 0;
      *sp = (*n > 1 || shard) ? *n : 0;
    }
  };

  // 3. scan units / partial slots / split tiles over the tiles, write the list.
  int32_t carry_u = 0, carry_s = 0, carry_f = 0;
  for (int32_t base = 0; base < T; base += 1024) {
    const int32_t t = base + tid;
    const int32_t P = t < T ? pages_of(t) : 0;
    int32_t n = 0, sp = 0;
    if (t < T) tile_units(t, P, &n, &sp);
    const int32_t f = (sp > 0 || (list_empty && t < T && P == 0)) ? 1 : 0;
    int32_t tu, ts, tf, eu, es, ef;
    block_exclusive_scan3(n, sp, f, s_scan, &eu, &es, &ef, &tu, &ts, &tf);
    eu += carry_u;
    es += carry_s;
    ef += carry_f;
    if (t < T) {
      if (cached) {
        s_ufirst[t] = eu;
        s_sfirst[t] = es;
      } else {
        for (int32_t u = 0; u < n && eu + u < p.ws.max_units; ++u) {
          int4 rec;
          rec.x = t;
          rec.y = unit_begin(P, n, u);
          rec.z = unit_begin(P, n, u + 1);
          rec.w = (n > 1 || shard) ? es + u : -1;
          p.ws.units[eu + u] = rec;
        }
      }
      p.ws.indptr[t] = es < p.ws.max_partials ? es : p.ws.max_partials;
      if (f) {
        // the same (clamped) range as indptr[t], indptr[t + 1]
        const int32_t mp = p.ws.max_partials;
        const int32_t r0 = es < mp ? es : mp, r1 = es + sp < mp ? es + sp : mp;
        p.ws.split_list[ef] = make_int4(t, r0, r1 - r0, 0);
      }
    }
    carry_u += tu;
    carry_s += ts;
    carry_f += tf;
  }
  // 4. unit records.  A fold plan writes them worker by worker (worker r:
  // its own tile, or the head of it, then the tail it takes over) together
  // with each worker's first unit.  Otherwise (cached case) one thread per
  // unit finds its tile by binary search over the first-unit offsets; with
  // more units than workers the queue is ordered longest unit first (a
  // counting sort over unit lengths; the order among units of equal length
  // is whatever the LDS atomics give, and does not change any result); the
  // attend kernel deals it to its workers in a snake, which pairs the longest
  // units of one pass with the shortest of the next the way a
  // longest-processing-time-first schedule would; with at most one unit per
  // worker every unit starts at once: tile order.
  if (fold) {
    __syncthreads();  // partial offsets of every tile
    const int32_t r = tid;
    const bool own = r < T && s_q[r] > 0, tail = r < p.G && r >= p.G - nl;
    int32_t total;
    const int32_t base = block_exclusive_scan((int32_t)own + (int32_t)tail, s_scan, &total);
    if (own) {
      const int32_t t = s_rt[r], P = s_q[r];
      p.ws.units[base] = r < nl ? make_int4(t, 0, cap, s_sfirst[t]) : make_int4(t, 0, P, -1);
    }
    if (tail) {
      const int32_t j = p.G - 1 - r, t = s_rt[j];
      p.ws.units[base + (int32_t)own] = make_int4(t, cap, s_q[j], s_sfirst[t] + 1);
    }
    if (r < p.G) hdr[kHdrWorkerTable + r] = base;
    if (r == 0) hdr[kHdrWorkerTable + p.G] = total;
  } else if (cached) {
    if (tid == 0) s_ufirst[T] = carry_u;
    for (int32_t i = tid; i <= kMaxUnitPages; i += 1024) s_lhist[i] = 0;
    __syncthreads();
    const int32_t NU = carry_u < p.ws.max_units ? carry_u : p.ws.max_units;
    auto unit_rec = [&](int32_t ug) {
      int32_t lo = 0, hi = T - 1;  // last tile with s_ufirst[t] <= ug
      while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (s_ufirst[mid] <= ug) lo = mid; else hi = mid - 1;
      }
      const int32_t t = lo, u = ug - s_ufirst[t];
      const int32_t P = s_pages[t];
      const int32_t n = s_ufirst[t + 1] - s_ufirst[t];
      const int32_t es = s_sfirst[t];
      int4 rec;
      rec.x = t;
      rec.y = unit_begin(P, n, u);
      rec.z = unit_begin(P, n, u + 1);
      rec.w = (n > 1 || shard) ? es + u : -1;
      return rec;
    };
    const bool lpt = NU > p.G;  // uniform
    // With query chunks the rows of a request read the same pages: the
    // queue keeps a request's units together (requests ordered by their
    // longest unit), unit index major, so that the rows of one page range sit
    // side by side and run on one XCD (see the attend kernel's dealing),
    // whose L2 serves the pages to every row.  Request b's range start sits
    // in s_q[b], its key in s_rt[b] (the fold plan's arrays, free here).
    const bool grouped = lpt && p.q_chunk > 1 && p.B <= kMaxWorkers && !shard;
    if (grouped) {
      for (int32_t b = tid; b < p.B; b += 1024) {
        const int32_t t0 = b * p.q_chunk, t1 = t0 + p.q_chunk;
        int32_t key = 0;
        for (int32_t t = t0; t < t1; ++t) {
          const int32_t n = s_ufirst[t + 1] - s_ufirst[t];
          if (n > 0) key = max(key, ceil_div(s_pages[t], n));
        }
        s_rt[b] = key;
        const int32_t cnt = s_ufirst[t1] - s_ufirst[t0];
        if (cnt > 0) atomicAdd(&s_lhist[key], cnt);  // 1 <= key <= kMaxUnitPages
      }
    } else {
      for (int32_t ug = tid; ug < NU; ug += 1024) {
        const int4 rec = unit_rec(ug);
        if (lpt) atomicAdd(&s_lhist[rec.z - rec.y], 1);  // 1 <= length <= kMaxUnitPages
        else p.ws.units[ug] = rec;
      }
    }
    __syncthreads();
    if (lpt) {
      // queue offset of each length: the number of longer units (thread i
      // takes length kMaxUnitPages - i)
      static_assert(kMaxUnitPages == 1024, "one thread per unit length");
      const int32_t len = kMaxUnitPages - tid;
      int32_t unused;
      s_lbase[len] = block_exclusive_scan(s_lhist[len], s_scan, &unused);
      __syncthreads();
      if (grouped) {
        for (int32_t b = tid; b < p.B; b += 1024) {
          const int32_t cnt = s_ufirst[(b + 1) * p.q_chunk] - s_ufirst[b * p.q_chunk];
          if (cnt > 0) s_q[b] = atomicAdd(&s_lbase[s_rt[b]], cnt);
        }
        __syncthreads();
        for (int32_t ug = tid; ug < NU; ug += 1024) {
          const int4 rec = unit_rec(ug);
          const int32_t b = rec.x / p.q_chunk, i = rec.x - b * p.q_chunk, u = ug - s_ufirst[rec.x];
          // rank in unit-major order: sum_r min(u, n_r) + #{r < i : n_r > u}
          int32_t rank = 0;
          for (int32_t r = 0; r < p.q_chunk; ++r) {
            const int32_t t = b * p.q_chunk + r, n = s_ufirst[t + 1] - s_ufirst[t];
            rank += min(u, n) + ((r < i && n > u) ? 1 : 0);
          }
          p.ws.units[s_q[b] + rank] = rec;
        }
      } else {
        for (int32_t ug = tid; ug < NU; ug += 1024) {
          const int4 rec = unit_rec(ug);
          p.ws.units[atomicAdd(&s_lbase[rec.z - rec.y], 1)] = rec;
        }
      }
    }
  }
  if (tid == 0) {
    p.ws.indptr[T] = carry_s;
    hdr[kHdrGrab] = 0;
    hdr[kHdrDone] = 0;
    hdr[kHdrUnits] = carry_u < p.ws.max_units ? carry_u : p.ws.max_units;
    hdr[kHdrPartials] = carry_s;
    hdr[kHdrChunk] = fold ? 0 : c;
    hdr[kHdrSplitTiles] = carry_f;
    hdr[kHdrTotalPages] = total_pages > INT32_MAX ? INT32_MAX : (int32_t)total_pages;
    // every split tile has at most this many parts
    hdr[kHdrMaxParts] = fold ? (nl > 0 ? 2 : 1) : (max_pages + c - 1) / c;
    hdr[kHdrSchedule] = fold ? p.G : 0;
    hdr[kHdrFoldCap] = fold ? cap : 0;
  }
}

// =============================================================== attend ===
//
// Work split inside a workgroup (4 waves, one per SIMD):
//  * S^T = K Q^T: wave w owns heads [32w, 32w+32) (its query fragment stays in
//    VGPRs) and computes their scores and softmax;
//  * P goes through LDS; O^T += V^T P^T: wave w owns output columns
//    [128w, 128w+128) for all 128 heads, so each wave transposes only a
//    quarter of V out of LDS.
//
// LDS layout of one staged step (32 cache rows): rows are cut into line
// groups of 128 B (bf16) or 64 B (fp8); group g of row r sits at
//   bf16: g*4096 + r*128 + ((c8 ^ ((r >> 1) & 7)) * 16)     (c8 = chunk in group)
//   fp8:  g*2048 + r*64  + ((c4 ^ swz4(r)) * 16),  swz4(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1)
// so every 1 KB direct-to-LDS instruction reads whole memory lines of 8 (16)
// rows, and the XOR spreads the operand reads over the LDS banks.  (fp8: the
// 16-byte slot of row r in a 256-byte bank period is 4 (r & 3) + (c4 ^
// swz4(r)); with bit 3 of the row in the XOR, the 32 rows of a K-fragment
// read fall two to a slot, the minimum, instead of four.)

//
// Latent rows (LAT: 656 B = 512 E4M3 codes at 0 | 4 fp32 tile scales at 512
// | 64 bf16 RoPE at 528): in LDS the latent's 8 line groups as fp8, then the
// RoPE as one bf16 line group at kRopeOff, then the rows' tile scales (16 B
// per row) at kData, and at kScaleT the same scales tile-major ([tile][row],
// written by wave 0 once its loads landed).
__device__ __forceinline__ uint32_t swz4(uint32_t r) { return ((r >> 1) & 3u) ^ ((r >> 3) & 1u); }

template <bool FP8, bool LAT = false>
struct StepLayout {
  static constexpr int kRowBytes = LAT ? 656 : FP8 ? kDimQK : 2 * kDimQK;   // 656 / 576 / 1152
  static constexpr int kRopeOff = 8 * kStepKeys * 64;                      // LAT: 16384
  static constexpr int kData = LAT ? kRopeOff + kStepKeys * 128 : kStepKeys * kRowBytes;  // 20480 / 18432 / 36864
  static constexpr int kScaleT = kData + 1024;                                            // LAT
  static constexpr int kBuf = LAT ? kData + 1536 : FP8 ? kData + 256 : kData;             // + fp32 scales
  // per wave and step (LAT: wave 0; waves 1-3 issue one fewer)
  static constexpr int kLoadsPerStep = LAT ? 6 : FP8 ? 5 : 9;
};

// Ring slots of the attend kernel: the step being multiplied (QK), the
// previous one (PV), and kDist steps in flight.  Four slots (two steps in
// flight) everywhere except the bf16 top-k variant, whose resolved pool rows
// take the LDS the fourth slot would need.
template <bool FP8, bool TOPK>
struct Ring {
  static constexpr int kSlots = (FP8 || !TOPK) ? 4 : 3;
  static constexpr int kDist = kSlots - 2;
};

// LDS map beyond the ring (bytes)
constexpr int kPBytes = kMaxHeads * kStepKeys * 2;   // P for all heads, bf16

// Placement of the 32 PV MFMAs of step j-1 in iteration j: kPV1 spread
// through the QK chain of step j, kPVTail after P of step j is written, and
// the last kPVDefer (column block 7) carried in registers past the next
// barrier, where they cover the latency of that iteration's first K-fragment
// reads; the softmax of step j rides on the rest.  Every accumulator keeps
// its order, so the results do not depend on these counts.
#ifndef SPLASH_PV1
#define SPLASH_PV1 0
#endif
#ifndef SPLASH_PV_TAIL
#define SPLASH_PV_TAIL 4
#endif
#ifndef SPLASH_PV_DEFER
#define SPLASH_PV_DEFER 2
#endif
constexpr int kPV1 = SPLASH_PV1, kPVTail = SPLASH_PV_TAIL, kPVDefer = SPLASH_PV_DEFER;
static_assert(kPV1 >= 0 && kPV1 <= 12 && kPVDefer >= 0 && kPVDefer <= 4 && kPVTail >= 0, "PV placement");

// Direct global->LDS loads, issued through asm so that the compiler's wait
// insertion (which cannot tell which LDS bytes they write) does not drain
// them before every LDS read; the kernel waits for them explicitly.  The
// source is a uniform 64-bit base plus a per-lane 32-bit offset; the LDS
// destination is M0 + 16 * lane (4 * lane for the dword form).  No
// instruction offset is used: it would move the LDS destination as well.
// M0 is restored afterwards.  NT: the non-temporal hint ("nt" on gfx950),
// which streams the lines through the caches instead of keeping them; the
// attend kernel sets it when no other tile reads the same pages (one query
// row per request), so that the cache rows do not evict what is reused.
#define SPLASH_DMA_ASM(INSN, ADDR, HINT, SREG)                                               \
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, " SREG "\n\ts_nop 0\n\t" INSN " %1, " ADDR HINT \
               "\n\ts_mov_b32 m0, %0"
template <bool NT>
__device__ __forceinline__ void dma_b128(const void* sbase, uint32_t voff, const uint8_t LDS_AS* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  uint32_t saved;
  if constexpr (NT)
    SPLASH_DMA_ASM("global_load_lds_dwordx4", "%2", " nt", "%3") : "=&s"(saved) : "v"(voff), "s"(sbase), "s"(m0) : "memory");
  else
    SPLASH_DMA_ASM("global_load_lds_dwordx4", "%2", "", "%3") : "=&s"(saved) : "v"(voff), "s"(sbase), "s"(m0) : "memory");
}
// The same loads from a per-lane 64-bit address (gathered rows anywhere in
// the pool).
template <bool NT>
__device__ __forceinline__ void dma_b128_v(uint64_t vaddr, const uint8_t LDS_AS* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  uint32_t saved;
  if constexpr (NT)
    SPLASH_DMA_ASM("global_load_lds_dwordx4", "off", " nt", "%2") : "=&s"(saved) : "v"(vaddr), "s"(m0) : "memory");
  else
    SPLASH_DMA_ASM("global_load_lds_dwordx4", "off", "", "%2") : "=&s"(saved) : "v"(vaddr), "s"(m0) : "memory");
}
template <bool NT>
__device__ __forceinline__ void dma_b32_v(uint64_t vaddr, const uint8_t LDS_AS* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  uint32_t saved;
  if constexpr (NT)
    SPLASH_DMA_ASM("global_load_lds_dword", "off", " nt", "%2") : "=&s"(saved) : "v"(vaddr), "s"(m0) : "memory");
  else
    SPLASH_DMA_ASM("global_load_lds_dword", "off", "", "%2") : "=&s"(saved) : "v"(vaddr), "s"(m0) : "memory");
}
template <bool NT>
__device__ __forceinline__ void dma_b32(const void* sbase, uint32_t voff, const uint8_t LDS_AS* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  uint32_t saved;
  if constexpr (NT)
    SPLASH_DMA_ASM("global_load_lds_dword", "%2", " nt", "%3") : "=&s"(saved) : "v"(voff), "s"(sbase), "s"(m0) : "memory");
  else
    SPLASH_DMA_ASM("global_load_lds_dword", "%2", "", "%3") : "=&s"(saved) : "v"(voff), "s"(sbase), "s"(m0) : "memory");
}

// Issue the direct-to-LDS loads of one step.
//  bf16: wave w loads rows [8w, 8w+8) of every line group g (t = g);
//  fp8:  instruction i = w + 4t (< 18) loads line group i >> 1, rows
//        [16 (i & 1), +16); waves 2 and 3 also load the 32 token scales.
//  LAT:  t < 4 as fp8 (the latent's 8 line groups); t = 4: wave w loads the
//        RoPE of rows [8w, 8w+8) into the bf16 layout; t = 5: wave 0 loads
//        the 32 rows' tile scales.
// step_src / step_scales are uniform; src_lane is the lane's byte offset
// inside the step for t = 0.
template <bool FP8, int t, bool LAT, bool NT>
__device__ __forceinline__ void issue_one(const uint8_t* __restrict__ step_src, const float* __restrict__ step_scales,
                                          uint32_t src_lane, uint8_t LDS_AS* buf, int wave) {
  if constexpr (LAT) {
    using L = StepLayout<true, true>;
    if constexpr (t < 4) {
      dma_b128<NT>(step_src + 128 * t, src_lane, buf + 4096 * t + 2048 * (wave >> 1) + 1024 * (wave & 1));
    } else {
      // lane id from an asm (volatile: recomputed here, not held in a
      // register across the loop), then the lane's source offset
      uint32_t ln;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
      if constexpr (t == 4) {
        const uint32_t r = 8 * wave + (ln >> 3);
        dma_b128<NT>(step_src, r * L::kRowBytes + 528 + (((ln & 7) ^ ((r >> 1) & 7)) * 16), buf + L::kRopeOff + 1024 * wave);
      } else if (wave == 0) {
        dma_b128<NT>(step_src, (ln & 31) * L::kRowBytes + 512, buf + L::kData);  // lanes 32-63 repeat 0-31
      }
    }
  } else if constexpr (!FP8) {
    dma_b128<NT>(step_src + 128 * t, src_lane, buf + 4096 * t + 1024 * wave);
  } else {
    if (t < 4 || wave + 4 * t < 18) {
      dma_b128<NT>(step_src + 128 * t, src_lane, buf + 4096 * t + 2048 * (wave >> 1) + 1024 * (wave & 1));
    } else {
      // byte offset of the lane's token scale, 4 (lane & 31), recomputed here
      // (volatile: not hoisted) rather than held in a register across the loop
      uint32_t voff;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_and_b32 %0, 31, %0\n\tv_lshlrev_b32 %0, 2, %0" : "=v"(voff));
      dma_b32<NT>(step_scales, voff, buf + 18432);
    }
  }
}

// Top-k variant: the lane's row of the step is a gathered pool row, at
// row_addr (its chunk included); its token scale (fp8, waves 2 and 3) at
// scale_addr.  Same LDS placement as issue_one.  LAT: the RoPE and tile-scale
// loads take other rows of the step than the latent ones; their pool rows
// are read here from step_rows (the step's 32 resolved rows in LDS), their
// bytes from the pool at kv.
template <bool FP8, int t, bool LAT, bool NT>
__device__ __forceinline__ void issue_one_v(uint64_t row_addr, uint64_t scale_addr, uint8_t LDS_AS* buf, int wave,
                                            const int32_t LDS_AS* step_rows, const uint8_t* kv) {
  if constexpr (LAT) {
    using L = StepLayout<true, true>;
    if constexpr (t < 4) {
      dma_b128_v<NT>(row_addr + 128 * t, buf + 4096 * t + 2048 * (wave >> 1) + 1024 * (wave & 1));
    } else {
      uint32_t ln;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
      const uint64_t base = (uint64_t)(uintptr_t)kv;
      if constexpr (t == 4) {
        const uint32_t r = 8 * wave + (ln >> 3);
        dma_b128_v<NT>(base + (uint64_t)(uint32_t)step_rows[r] * L::kRowBytes + 528 + (((ln & 7) ^ ((r >> 1) & 7)) * 16),
                   buf + L::kRopeOff + 1024 * wave);
      } else if (wave == 0) {
        dma_b128_v<NT>(base + (uint64_t)(uint32_t)step_rows[ln & 31] * L::kRowBytes + 512, buf + L::kData);
      }
    }
  } else if constexpr (!FP8) {
    dma_b128_v<NT>(row_addr + 128 * t, buf + 4096 * t + 1024 * wave);
  } else {
    if (t < 4 || wave + 4 * t < 18)
      dma_b128_v<NT>(row_addr + 128 * t, buf + 4096 * t + 2048 * (wave >> 1) + 1024 * (wave & 1));
    else
      dma_b32_v<NT>(scale_addr, buf + 18432);
  }
}
template <bool FP8, bool LAT, bool NT, int t = 0>
__device__ __forceinline__ void issue_from_v(uint64_t row_addr, uint64_t scale_addr, uint8_t LDS_AS* buf, int wave,
                                             const int32_t LDS_AS* step_rows, const uint8_t* kv) {
  if constexpr (t < StepLayout<FP8, LAT>::kLoadsPerStep) {
    issue_one_v<FP8, t, LAT, NT>(row_addr, scale_addr, buf, wave, step_rows, kv);
    issue_from_v<FP8, LAT, NT, t + 1>(row_addr, scale_addr, buf, wave, step_rows, kv);
  }
}

template <bool FP8, bool LAT, bool NT, int t = 0>
__device__ __forceinline__ void issue_from(const uint8_t* __restrict__ step_src, const float* __restrict__ step_scales,
                                           uint32_t src_lane, uint8_t LDS_AS* buf, int wave) {
  if constexpr (t < StepLayout<FP8, LAT>::kLoadsPerStep) {
    issue_one<FP8, t, LAT, NT>(step_src, step_scales, src_lane, buf, wave);
    issue_from<FP8, LAT, NT, t + 1>(step_src, step_scales, src_lane, buf, wave);
  }
}

template <bool FP8, bool LAT, bool NT>
__device__ __forceinline__ void issue_step(const uint8_t* __restrict__ step_src, const float* __restrict__ step_scales,
                                           uint32_t src_lane, uint8_t LDS_AS* buf, int wave) {
  issue_from<FP8, LAT, NT>(step_src, step_scales, src_lane, buf, wave);
}

// QK^T MFMAs are issued through inline asm with a VGPR accumulator: the
// compiler picks one MFMA destination class per function, and the output
// accumulator already fills the 256 accumulation registers.  The QK^T of a
// step is one accumulation chain: every MFMA adds into exactly the registers
// the previous one wrote, which the matrix pipe forwards without wait states;
// wait_mfma_vgpr() covers the latency before VALU code reads the result.
template <bool FIRST, bool VALU_SRC>
__device__ __forceinline__ void mfma_qk(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  if constexpr (FIRST) {
    if constexpr (VALU_SRC)
      asm volatile("s_nop 2\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=v"(acc) : "v"(a), "v"(b));
    else
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=v"(acc) : "v"(a), "v"(b));
  } else {
    if constexpr (VALU_SRC)
      asm volatile("s_nop 2\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "v"(b));
    else
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "v"(b));
  }
}

__device__ __forceinline__ void wait_mfma_vgpr(f32x16& acc) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc));
}

// K operand fragment ks (A operand: lane = key row n32, 8 dims).
template <bool FP8>
__device__ __forceinline__ bf16x8 load_k_frag(const uint8_t LDS_AS* buf, const uint32_t* kbase, int ks) {
  if constexpr (!FP8) {
    return *(const bf16x8 LDS_AS*)(buf + kbase[ks & 3] + 4096 * (ks >> 2));
  } else {
    const u32x2 raw = *(const u32x2 LDS_AS*)(buf + kbase[ks & 3] + 2048 * (ks >> 2));
    return fp8x8_to_bf16(raw);
  }
}

// V^T operand fragment (column block cb, key half kh) via transposing reads.
template <bool FP8>
__device__ __forceinline__ bf16x8 load_v_frag(const uint8_t LDS_AS* buf, const uint32_t (*vbase)[2], int cb, int kh) {
  if constexpr (!FP8) {
    const uint8_t LDS_AS* p = buf + 4096 * (cb >> 1) + 2048 * kh;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((s16x4 LDS_AS*)(p + vbase[cb & 1][0]));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((s16x4 LDS_AS*)(p + vbase[cb & 1][1]));
    const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
    return __builtin_bit_cast(bf16x8, (u32x4){l2[0], l2[1], h2[0], h2[1]});
  } else {
    const i32x2 raw = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
        (i32x2 LDS_AS*)(buf + vbase[cb & 1][0] + 2048 * (cb >> 1) + 1024 * kh));
    return fp8x8_to_bf16(__builtin_bit_cast(u32x2, raw));
  }
}

// Operand fragments as the LDS reads return them (fp8: the 8 codes) and
// their conversion to the MFMA's bf16.  The stream converts a fragment in
// the slot that uses it, so the read has the slots since its issue to land;
// converting right at the read would wait for it there.
template <bool FP8>
using FragRaw = typename std::conditional<FP8, u32x2, bf16x8>::type;
template <bool FP8>
__device__ __forceinline__ FragRaw<FP8> load_k_raw(const uint8_t LDS_AS* buf, const uint32_t* kbase, int ks) {
  if constexpr (!FP8) return *(const bf16x8 LDS_AS*)(buf + kbase[ks & 3] + 4096 * (ks >> 2));
  else return *(const u32x2 LDS_AS*)(buf + kbase[ks & 3] + 2048 * (ks >> 2));
}
template <bool FP8>
__device__ __forceinline__ FragRaw<FP8> load_v_raw(const uint8_t LDS_AS* buf, const uint32_t (*vbase)[2], int cb,
                                                   int kh) {
  if constexpr (!FP8) {
    return load_v_frag<false>(buf, vbase, cb, kh);
  } else {
    const i32x2 raw = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
        (i32x2 LDS_AS*)(buf + vbase[cb & 1][0] + 2048 * (cb >> 1) + 1024 * kh));
    return __builtin_bit_cast(u32x2, raw);
  }
}
template <bool FP8>
__device__ __forceinline__ bf16x8 frag_bf16(const FragRaw<FP8>& r) {
  if constexpr (FP8) return fp8x8_to_bf16(r);
  else return r;
}

// Latent rows: 8 E4M3 codes of one latent tile times the tile's scale.  The
// conversion applies only the scale operand's exponent (2^floor(log2 s)),
// which is why the format requires power-of-two scales; the products are
// then exact in bf16.
__device__ __forceinline__ bf16x8 fp8x8_scaled_to_bf16(u32x2 raw, float scale) {
  u32x4 r;
  r[0] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[0], scale, false));
  r[1] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[0], scale, true));
  r[2] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[1], scale, false));
  r[3] = __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)raw[1], scale, true));
  return __builtin_bit_cast(bf16x8, r);
}

// Latent rows: a wave's PV covers output columns [128 wave, +128), one
// latent tile, so the tile scale of each key multiplies that key's P weight
// instead of V.  The scales are powers of two 2^e, so the product is the
// weight with e added to its bf16 exponent field: one packed 16-bit add per
// pair of weights (d holds e << 7 of both keys), and a packed max that
// turns an exponent pushed below the normal range into 0.  Exact while the
// result stays normal: weights are at most 2^64 in the pass that is kept
// and e <= 63 (a scale above 2^63 is outside the format); a weight pushed
// below 2^-126 contributes nothing the fp32 sum would keep.
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef short i16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16x8 scale_p(bf16x8 p, const u32x4& d) {
  const u32x4 w = __builtin_bit_cast(u32x4, p);
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // (scalar copies first: a bit cast taken straight from a vector element
    // reads element 0 whatever the index)
    const unsigned wi = w[i], di = d[i];
    const u16x2 sum = __builtin_bit_cast(u16x2, wi) + __builtin_bit_cast(u16x2, di);
    r[i] = __builtin_bit_cast(unsigned, __builtin_elementwise_max(__builtin_bit_cast(i16x2, sum), (i16x2){0, 0}));
  }
  return __builtin_bit_cast(bf16x8, r);
}

// Latent rows: the exponent steps (e << 7, 16 bits per key) of the tile-`wave`
// scales of the 8 keys of the P^T fragment (key half kh) a lane reads;
// element e is key 16kh + 8(e >> 2) + 4h + (e & 3) (the slot order of the P
// exchange), so the four key pairs are two 8-byte reads of the tile-major
// table ([tile][key], 2 bytes each).
__device__ __forceinline__ void load_p_scales(const uint8_t LDS_AS* scales_t, int kh, int h, int wave, u32x4& d) {
  const uint8_t LDS_AS* base = scales_t + 2 * (32 * wave + 16 * kh + 4 * h);
  const u32x2 a = *(const u32x2 LDS_AS*)base, b = *(const u32x2 LDS_AS*)(base + 16);
  d = (u32x4){a[0], a[1], b[0], b[1]};
}

// P^T operand fragment (head block hb, key half kh) from the P exchange area:
// head hh's 32 weights are 64 B, slot (kh, half) at ((2kh + half) ^ (hh>>2 & 3)) * 16.
__device__ __forceinline__ uint32_t p_slot(uint32_t hh, uint32_t kh, uint32_t half) {
  return hh * 64 + (((2 * kh + half) ^ ((hh >> 2) & 3)) * 16);
}

// PV of one 32-key step as a standalone MFMA stream (the unit's last step,
// which has no QK to interleave with): 32 MFMAs,
// o[cbl][hb] += V^T(cb = 4*wave + cbl, kh) P^T(hb, kh) with V from `vbuf` and
// P from the P exchange area (LAT: P scaled by the keys' tile scales, whose
// tile-major copy sits at vbuf + lat_scales).
template <bool FP8, bool LAT = false>
__device__ __forceinline__ void pv_stream(const uint8_t LDS_AS* vbuf, const uint32_t (*vbase)[2],
                                          const uint8_t LDS_AS* p_lds, int wave, int n32, int h,
                                          f32x16 (&o)[4][4], int lat_scales, const bf16x8& dv,
                                          const bf16x8 (&dp)[4]) {
  // the previous step's deferred MFMAs (column block 7)
#pragma unroll
  for (int hb = 4 - kPVDefer; hb < 4; ++hb) o[3][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dv, dp[hb], o[3][hb], 0, 0, 0);
  // V fragments are double-buffered one column block ahead (c = 4kh + cbl).
  bf16x8 pf[4], vf[2];
  u32x4 psc;
  if constexpr (LAT) load_p_scales(vbuf + lat_scales, 0, h, wave, psc);
#pragma unroll
  for (int hb = 0; hb < 4; ++hb) {
    pf[hb] = *(const bf16x8 LDS_AS*)(p_lds + p_slot(32 * hb + n32, 0, h));
    if constexpr (LAT) pf[hb] = scale_p(pf[hb], psc);
  }
  if constexpr (LAT) load_p_scales(vbuf + lat_scales, 1, h, wave, psc);
  vf[0] = load_v_frag<FP8>(vbuf, vbase, 4 * wave, 0);
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    // prefetch the V fragment of the next column block before the MFMAs of
    // this one
    if ((i & 3) == 0 && i < 28) {
      const int cn = (i >> 2) + 1;
      vf[cn & 1] = load_v_frag<FP8>(vbuf, vbase, 4 * wave + (cn & 3), cn >> 2);
    }
    const int c = i >> 2, kh = i >> 4, cbl = (i >> 2) & 3, hb = i & 3;
    o[cbl][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[c & 1], pf[hb], o[cbl][hb], 0, 0, 0);
    // P fragments of key half 1 replace those of half 0 once the last MFMA
    // of half 0 that reads them has been issued
    if (kh == 0 && cbl == 3) {
      pf[hb] = *(const bf16x8 LDS_AS*)(p_lds + p_slot(32 * hb + n32, 1, h));
      if constexpr (LAT) pf[hb] = scale_p(pf[hb], psc);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// TOPK: the top-k variant.  Row n attends the first topk_count[n] token
// positions of its list topk_idx[n] (of request b = n / q_chunk); a unit
// covers list entries [64 p0, 64 p1) instead of pages, and its prologue
// resolves every entry to its pool row (into the LDS the block-table slice
// uses otherwise), from which each lane loads its staged row.
// LAT: the fp8 latent-row cache (FP8 set too): latent tiles with their tile
// scale for QK, the RoPE read as bf16, and for PV each wave's P scaled by its
// tile's key scales.
// NT: non-temporal cache-row loads and result stores (one query row per
// request).  Q8 (fp8 caches): QK on the fp8 matrix pipe (split query, K's
// own codes); without it K is converted to bf16 for the bf16 MFMA.
template <bool FP8, bool TOPK, bool LAT, bool NT, bool Q8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attend_kernel(AttendLaunch a) {
  static_assert(!LAT || FP8, "latent rows are an fp8 variant");
  static_assert(!Q8 || FP8, "the fp8-pipe QK serves the fp8 caches");
  using L = StepLayout<FP8, LAT>;
  constexpr int kSlots = Ring<FP8, TOPK>::kSlots, kDist = Ring<FP8, TOPK>::kDist;
  constexpr int kRing = kSlots * L::kBuf;
  // Unit overlap (dense caches): the next unit's query and first kDist
  // steps are issued before this unit's epilogue stores, so their latency
  // hides behind the epilogue.
  constexpr bool kOverlap = !TOPK && !LAT;
  // LDS map: the ring, then the P exchange area (two steps), then (top-k
  // only) the unit's resolved pool rows.  The dense variants read their page
  // ids from the block table in memory through the scalar cache, which is
  // what lets the bf16 ring hold four 36-KB steps in the 160 KB.  The
  // epilogue stages its rows, followed by the per-head normaliser, in LDS
  // idle at that time: for bf16 in ring slots 0-1, with a unit's step j in
  // slot (j + 2) mod 4 so that the next unit's first two steps land in slots
  // 2-3 meanwhile; for fp8 after the P area; otherwise anywhere in the ring.
  constexpr int kPOff = kRing;
  constexpr int kBtOff = kPOff + 2 * kPBytes;
  constexpr int kStageRow = 128 * 4 + 16;            // epilogue: bytes per head, padded off the banks
  constexpr int kLOff = 4 * 32 * kStageRow;          // epilogue: per-head normaliser, 128 floats
  constexpr int kScOff = kLOff + kMaxHeads * 4;      // epilogue: per wave, the normalisers times each
                                                     // head's quarter scale (split partials)
  constexpr int kStageBytes = kScOff + 4 * kMaxHeads * 4;
  constexpr int kStageOff = (kOverlap && FP8) ? kBtOff : 0;
  constexpr int kSlotBase = (kOverlap && !FP8) ? 2 : 0;
  static_assert(!(kOverlap && !FP8) || kStageBytes <= 2 * L::kBuf, "bf16 staging fits in ring slots 0-1");
  static_assert(kStageOff > 0 || kStageBytes <= kRing, "staging fits in the ring");
  constexpr int kSmemA = kBtOff + (TOPK ? kTopkUnitPages * kPage * 4 : 0);
  constexpr int kSmem = kSmemA > kStageOff + kStageBytes ? kSmemA : kStageOff + kStageBytes;
  static_assert(kSmem <= 163840, "LDS budget");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmem];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int h = lane >> 5, n32 = lane & 31;
  // QK and softmax role: head block `wave` (32 heads) over all 576 dims
  const int head = 32 * wave + n32;
  const bool head_ok = head < a.H;
  const float c2 = a.softmax_scale * 1.4426950408889634f;  // log2(e)
  // fp8 caches (Q8): QK on the fp8 matrix pipe with the query split in two
  // E4M3 terms; its power-of-two row scale joins the softmax constant
  constexpr bool kQ8 = Q8;
  constexpr int kQB = LAT ? 8 : 9;  // 64-dim blocks on the fp8 pipe (latent rows: the RoPE 64 stay bf16)
  float c2v = c2;
  // block scales of the fp8 QK MFMAs (E8M0): 1, and 2^-4 for the lo terms
  const int bs_one = (int)opaque(127u), bs_lo = (int)opaque(127u - 4u);
  const uint8_t* __restrict__ kv = (const uint8_t*)a.kv;
  uint8_t LDS_AS* sm = (uint8_t LDS_AS*)smem;
  uint8_t LDS_AS* p_lds = sm + kPOff;
  float LDS_AS* l_lds = (float LDS_AS*)(sm + kStageOff + kLOff);
  int32_t LDS_AS* s_bt = (int32_t LDS_AS*)(sm + kBtOff);  // top-k only

  // ---- per-lane offsets (bytes), fixed for the kernel ----
  uint32_t src_lane, dma_row, dma_slot;
  if constexpr (!FP8) {
    dma_row = 8 * wave + (lane >> 3);
    src_lane = dma_row * 1152 + (((lane & 7) ^ ((dma_row >> 1) & 7)) * 16);
    dma_slot = 1024 * wave + 16 * lane;              // + 4096 t
  } else {
    dma_row = 16 * (wave & 1) + (lane >> 2);
    src_lane = dma_row * L::kRowBytes + 64 * (wave >> 1) + (((lane & 3) ^ swz4(dma_row)) * 16);
    dma_slot = 2048 * (wave >> 1) + 1024 * (wave & 1) + 16 * lane;   // + 4096 t
  }
  // K operand of k-step ks (dims 16ks + 8h + [0, 8)): row n32, chunk
  // 2(ks & 3) + h of line group ks >> 2 (bf16), or 16-byte chunk ks & 3, half
  // h (fp8); kbase[ks & 3] + G * (ks >> 2) addresses it (G = group stride).
  // LAT: the RoPE k-steps 32..35 read the bf16 line group at kRopeOff
  // through kbase_r (the bf16 formula).
  uint32_t kbase[4], kbase_r[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    if constexpr (!FP8)
      kbase[m] = n32 * 128 + (((2 * m + h) ^ ((n32 >> 1) & 7)) * 16);
    else
      kbase[m] = n32 * 64 + ((m ^ swz4(n32)) * 16) + 8 * h;
    kbase_r[m] = L::kRopeOff + n32 * 128 + (((2 * m + h) ^ ((n32 >> 1) & 7)) * 16);
  }
  // V operand (transposing reads), see load_v_frag
  const int i16 = lane & 15, g16 = lane >> 4;
  uint32_t vbase[2][2];
  if constexpr (!FP8) {
    // source lane: row 16kh + 8t + 4h + (i16>>2), chunk 4cb + cc, 8*(i16&1) bytes in
    const uint32_t cc = 2 * (g16 & 1) + ((i16 >> 1) & 1);
    const uint32_t rb = 4 * h + (i16 >> 2);
#pragma unroll
    for (int cbo = 0; cbo < 2; ++cbo)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const uint32_t row = 8 * t + rb;
        vbase[cbo][t] = row * 128 + (((4 * cbo + cc) ^ ((row >> 1) & 7)) * 16) + 8 * (i16 & 1);
      }
  } else {
    // tr8 source lane: key k = i16>>1 of the slot order, 8 columns at
    // 32cb + 16(g16&1) + 8(i16&1), i.e. 16-byte chunk 2cb + (g16&1)
    const int k = i16 >> 1;
    const uint32_t rowk = 8 * (k >> 2) + 4 * h + (k & 3);
#pragma unroll
    for (int cbo = 0; cbo < 2; ++cbo) {
      const uint32_t c4 = 2 * cbo + (g16 & 1);
      vbase[cbo][0] = rowk * 64 + ((c4 ^ swz4(rowk)) * 16) + 8 * (i16 & 1);  // rowk < 16: swz4 is that of rowk + 16
      vbase[cbo][1] = 0;
    }
  }

  // Schedule, without atomics so that a worker knows its next unit ahead:
  // under a fold plan made for this many workers, worker g runs its own
  // units [table[g], table[g + 1]); otherwise the queue, ordered longest unit
  // first, is dealt in a snake (pass k gives worker g position kG + g, or
  // kG + G-1-g on odd passes), which pairs the longest units of one pass with
  // the shortest of the next as a longest-first greedy schedule would.  The
  // plan, the records and the lengths are read through the scalar cache:
  // nothing writes them while the kernel runs.
  typedef const int32_t __attribute__((address_space(4))) ConstI32;
  typedef const i32x4 __attribute__((address_space(4))) ConstI32x4;
  ConstI32* hdr = (ConstI32*)a.ws.header;
  const int32_t G = (int32_t)gridDim.x, g = (int32_t)blockIdx.x;
  const bool own_run = hdr[kHdrSchedule] == G;
  const int32_t run_begin = own_run ? hdr[kHdrWorkerTable + g] : 0;
  const int32_t run_end = own_run ? hdr[kHdrWorkerTable + g + 1] : hdr[kHdrUnits];
  // With query chunks, the rows of one request read the same pages: the
  // queue's neighbours (the longest-first order keeps a request's units
  // together) go to workers of one XCD, whose L2 then serves the pages to
  // all of them.  Workgroups are placed on the 8 XCDs round robin, so
  // queue slot l of a pass goes to worker (l mod G/8) * 8 + l / (G/8).
  const int32_t lg = (a.q_chunk > 1 && (G & 7) == 0) ? (g & 7) * (G >> 3) + (g >> 3) : g;
  auto unit_rec = [&](int k) -> i32x4 {
    const int32_t u = own_run ? run_begin + k : k * G + ((k & 1) ? G - 1 - lg : lg);
    if (u < run_end) return ((ConstI32x4*)a.ws.units)[u];
    return (i32x4){-1, 0, 0, 0};
  };
  // A unit's keys: request b, pages [p0, p1) (a shard's count from its first
  // page), keys [key_begin, key_end) in nsteps steps of 32.
  struct Geo {
    int tile, slot, b, p0, p1, key_begin, key_end, nsteps;
  };
  auto geometry = [&](const i32x4 r) {
    Geo u;
    u.tile = r.x;
    u.slot = r.w;
    u.b = r.x / a.q_chunk;
    const int qi = r.x - u.b * a.q_chunk;
    int Lk = tile_keys(((ConstI32*)a.seq_lens)[u.b], a.q_chunk, qi);
    u.p0 = r.y;
    u.p1 = r.z;
    if (a.key_end) {
      const int first = ((ConstI32*)a.key_begin)[u.b] >> 6;
      u.p0 += first;
      u.p1 += first;
      Lk = min(Lk, ((ConstI32*)a.key_end)[u.b]);
    }
    if constexpr (TOPK) Lk = ((ConstI32*)a.topk_count)[r.x];  // entries of the row's list
    u.key_begin = u.p0 * kPage;
    u.key_end = min(u.p1 * kPage, Lk);
    u.nsteps = (u.key_end - u.key_begin + kStepKeys - 1) / kStepKeys;
    return u;
  };
  // Query fragments: B operands, k = dims 16ks + 8h + [0, 8), row = head.
  // Padding heads (head >= H) take head 0's row: their scores stay finite and
  // nothing of theirs is stored.  (Nothing consumes the loaded values here,
  // so the loads stay in flight until the first QK MFMA.)
  // (kQ8: fragments 2m and 2m + 1 side by side in q8[m]; after
  // split_query, q8[2kb] holds the hi codes of dims block kb, q8[2kb + 1] the
  // lo codes, in the byte order of the fp8 K operand)
  bf16x8 qf[kQ8 ? 1 : 36];
  i32x8 q8[kQ8 ? 2 * kQB : 1];
  bf16x8 qr[LAT ? 4 : 1];  // latent rows: the RoPE fragments 32-35, bf16 (times the row scale's inverse)
  auto load_q = [&](int t) {
    const uint16_t* qrow = (const uint16_t*)a.q + ((size_t)t * a.H + (head_ok ? head : 0)) * kDimQK + 8 * h;
    if constexpr (kQ8) {
#pragma unroll
      for (int m = 0; m < 2 * kQB; ++m) {
        const u32x4 f0 = *(const u32x4*)(qrow + 32 * m), f1 = *(const u32x4*)(qrow + 32 * m + 16);
        q8[m] = __builtin_bit_cast(i32x8, __builtin_shufflevector(f0, f1, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      if constexpr (LAT) {
#pragma unroll
        for (int p = 0; p < 4; ++p) qr[p] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qrow + 16 * (32 + p)));
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < 36; ++ks) qf[ks] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qrow + 16 * ks));
    }
  };
  // kQ8: the head's row scale (lanes l and l ^ 32 hold its two halves), then
  // the split of every block; sets the lane's softmax constant
  auto split_query = [&]() {
    auto bmax = [](float m, uint32_t w) {
      return fmaxf(m, fmaxf(fabsf(__uint_as_float(w << 16)), fabsf(__uint_as_float(w & 0xFFFF0000u))));
    };
    float mx = 0.f;
#pragma unroll
    for (int m = 0; m < 2 * kQB; ++m)
#pragma unroll
      for (int d = 0; d < 8; ++d) mx = bmax(mx, (uint32_t)q8[m][d]);
    if constexpr (LAT) {
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int d = 0; d < 4; ++d) mx = bmax(mx, __builtin_bit_cast(u32x4, qr[p])[d]);
    }
    mx = fmaxf(mx, wave_xor32(mx));
    int e = (int)((__float_as_uint(mx) >> 23) & 255u) - 127;  // floor(log2 max), -127 for 0
    // (every finite bf16 has e <= 127, so the largest scaled value stays
    // under 256; rows below 2^-100 become zeros, their scores ~0 anyway)
    e = e < -100 ? -100 : (e > 127 ? 127 : e);
    const float inv = __uint_as_float((uint32_t)(127 + 7 - e) << 23);  // 2^(7 - e)
    c2v = c2 * __uint_as_float((uint32_t)(127 - 7 + e) << 23);         // c2 * 2^(e - 7)
#pragma unroll
    for (int kb = 0; kb < kQB; ++kb) split_query_block(q8[2 * kb], q8[2 * kb + 1], inv);
    if constexpr (LAT) {
      // the RoPE fragments times the same power of two (exact in bf16)
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const u32x4 w = __builtin_bit_cast(u32x4, qr[p]);
        u32x4 o;
#pragma unroll
        for (int d = 0; d < 4; ++d)
          o[d] = pack_bf16x2(__uint_as_float(w[d] << 16) * inv, __uint_as_float(w[d] & 0xFFFF0000u) * inv);
        qr[p] = __builtin_bit_cast(bf16x8, o);
      }
    }
  };

  i32x4 cur = unit_rec(0), nxt = unit_rec(1);
  bool pre = false;  // the current unit's query and first steps were issued by the previous unit
  for (int k = 0; cur.x >= 0; ++k) {
    const Geo U = geometry(cur);
    const int tile = U.tile, slot = U.slot, b = U.b, p0 = U.p0, p1 = U.p1;
    const int key_begin = U.key_begin, key_end = U.key_end, nsteps = U.nsteps;
    // the record after next, and what the next unit needs at this unit's
    // end, read now (scalar loads) and used there
    const i32x4 nxt2 = unit_rec(k + 2);
    Geo N = {};
    int n_phys = 0;
    if (kOverlap && nxt.x >= 0) {
      N = geometry(nxt);
      n_phys = ((ConstI32*)a.block_table)[(size_t)N.b * a.bt_stride + N.p0];
    }

    if constexpr (TOPK) {
      // pool row of every list entry of the unit (entries past the list end
      // read pool row 0, whose keys the tail mask removes)
      const int32_t* sel = a.topk_idx + (size_t)tile * a.topk;
      const int32_t* btr = a.block_table + (size_t)b * a.bt_stride;
      for (int e = tid; e < (p1 - p0) * kPage; e += 256) {
        int row = 0;
        if (key_begin + e < key_end) {
          const int pos = sel[key_begin + e];
          row = btr[pos >> 6] * kPage + (pos & (kPage - 1));
        }
        s_bt[e] = row;
      }
    }
    // dense variants: the unit's block-table entries, read through the
    // scalar cache (the table is not written while the kernel runs)
    ConstI32* bt_unit = (ConstI32*)(a.block_table + (size_t)b * a.bt_stride + p0);

    if (!pre) load_q(tile);
    __syncthreads();  // (top-k) the resolved rows visible

    auto step_src = [&](int j, int phys) {
      const int key = key_begin + j * kStepKeys;
      return kv + (size_t)phys * (kPage * L::kRowBytes) + (size_t)((key >> 5) & 1) * (kStepKeys * L::kRowBytes);
    };
    auto step_scales = [&](int j, int phys) -> const float* {
      if constexpr (!FP8 || LAT) return nullptr;
      const int key = key_begin + j * kStepKeys;
      return a.kv_scales + (size_t)phys * kPage + ((key >> 5) & 1) * kStepKeys;
    };
    // page of step j (two steps per page: key_begin is a page boundary)
    auto step_phys = [&](int j) { return bt_unit[j >> 1]; };
    // top-k: pool row of the lane's staged row of step j, and (fp8) of the
    // token scale it loads; their addresses
    auto lane_row = [&](int j) { return s_bt[j * kStepKeys + dma_row]; };
    auto scale_row = [&](int j) { return FP8 ? s_bt[j * kStepKeys + (lane & 31)] : 0; };
    auto row_addr = [&](int r) {
      return (uint64_t)(uintptr_t)kv + (uint64_t)(uint32_t)r * L::kRowBytes + (src_lane - dma_row * L::kRowBytes);
    };
    auto scale_addr = [&](int r) { return (uint64_t)(uintptr_t)a.kv_scales + (uint64_t)(uint32_t)r * 4; };
    // ring slot of step j; the offset is laundered so the compiler keeps one
    // scalar per step instead of deriving per-lane induction variables
    auto slot_buf = [&](int j) {
      uint32_t off = (uint32_t)((j + kSlotBase) % kSlots) * L::kBuf;
      asm volatile("" : "+s"(off));
      return sm + off;
    };

    // Softmax reference: fixed at the first step's max (O is still zero
    // there), never moved afterwards, so O is never rescaled inside the loop.
    // If a later logit exceeds it by more than 64 (base 2), P could overflow:
    // the workgroup then redoes the unit with the unit's true max, which is
    // known after the first pass.
    float m_init = -INFINITY;
    f32x16 o[4][4];  // [column block cb - 4*wave][head block]
    bf16x8 d_v, d_p[4];  // operands of the PV MFMAs carried past a barrier
    float m_ref, l_run, l_exact;
    for (int pass = 0;; ++pass) {
      // Pipeline: step j is staged kDist steps ahead; iteration j runs QK of
      // step j together with PV of step j-1, then the softmax of step j.
#pragma unroll
      for (int j = 0; j < kDist; ++j)
        if (j < nsteps && (pass > 0 || !pre)) {
          if constexpr (TOPK) {
            issue_from_v<FP8, LAT, NT>(row_addr(lane_row(j)), scale_addr(scale_row(j)), slot_buf(j), wave,
                                   s_bt + j * kStepKeys, kv);
          } else {
            const int ph = step_phys(j);
            issue_step<FP8, LAT, NT>(step_src(j, ph), step_scales(j, ph), src_lane, slot_buf(j), wave);
          }
        }
      if constexpr (kQ8) {
        if (pass == 0) split_query();
      }

#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) o[x][y] = (f32x16){};
      m_ref = m_init;
      d_v = (bf16x8){};
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) d_p[hb] = (bf16x8){};
      l_run = 0.f;
      l_exact = 0.f;
      float tmax = -INFINITY;  // largest t = z*log2(e) - m_ref of this pass, per lane

      // page of the step staged next (dense): read one iteration early
      int next_phys = !TOPK && kDist < nsteps ? step_phys(kDist) : 0;
      // top-k: the rows of the step staged next (per lane), read from LDS one
      // iteration early
      int next_row = TOPK && kDist < nsteps ? lane_row(kDist) : 0;
      int next_srow = TOPK && kDist < nsteps ? scale_row(kDist) : 0;
      // One pipeline iteration: staging wait, QK of step j (interleaved with
      // part of PV of step j-1 and the loads of step j + kDist), then the
      // softmax of step j interleaved with the rest of PV of step j-1.
      // pf_mode 1 (the steady state): step j + kDist exists, so it is staged
      // here, and step j is not the last one (no history end inside it); 2:
      // nothing left to stage; 0 (the first step): decided at run time.
      auto qk_softmax = [&](int j, auto with_pv, auto pf_mode) {
        constexpr bool kPV = decltype(with_pv)::value;
        constexpr int kPFM = decltype(pf_mode)::value;
        uint8_t LDS_AS* buf = slot_buf(j);                     // step j
        uint8_t LDS_AS* vbuf = slot_buf(j + kSlots - 1);       // step j-1
        const uint8_t LDS_AS* p_prev = p_lds + kPBytes * ((j + 1) & 1);  // P of step j-1
        const int key0 = key_begin + j * kStepKeys;
        const int valid = key_end - key0;  // >= 1; >= 32 in the steady state
        const bool pf_next = kPFM == 1 ? true : kPFM == 2 ? false : (j + kDist < nsteps);
        const bool may_end = kPFM != 1;
        const int pf_phys = TOPK ? 0 : next_phys;
        const uint8_t* pf_src = step_src(j + kDist, pf_phys);
        const float* pf_scales = step_scales(j + kDist, pf_phys);
        uint64_t pf_row = 0, pf_srow = 0;
        const int32_t LDS_AS* pf_rows = s_bt + (j + kDist) * kStepKeys;  // top-k: rows of step j + kDist
        if constexpr (TOPK) {
          pf_row = row_addr(next_row);
          pf_srow = scale_addr(next_srow);
        }
        uint8_t LDS_AS* pf_buf = slot_buf(j + kDist);
        if (kDist == 2 && (kPFM == 1 || j + 1 < nsteps)) {
          // step j + 1's loads may still be in flight (LAT: only wave 0 loads
          // the tile scales)
          if (LAT && wave != 0) wait_vmcnt<L::kLoadsPerStep - 1>();
          else wait_vmcnt<L::kLoadsPerStep>();
        } else {
          wait_vmcnt<0>();
        }
        if (may_end && valid < kStepKeys) {
          // rows past the history end: P is zero there, V must not be NaN
          const u32x4 z = {0, 0, 0, 0};
          if ((int)opaque(dma_row) >= valid) {
#pragma unroll
            for (int t = 0; t < L::kLoadsPerStep; ++t)
              if (!FP8 || t < 4 || (!LAT && wave + 4 * t < 18)) *(u32x4 LDS_AS*)(buf + dma_slot + 4096 * t) = z;
          }
          if constexpr (LAT) {
            // their RoPE and tile scales (each cleared by the wave that
            // loaded it, after its own loads landed): zero scales keep the
            // scaled P and K finite
            if ((int)opaque(8 * wave + (lane >> 3)) >= valid)
              *(u32x4 LDS_AS*)(buf + L::kRopeOff + 1024 * wave + 16 * lane) = z;
            if (wave == 0 && (int)(lane & 31) >= valid) *(u32x4 LDS_AS*)(buf + L::kData + 16 * lane) = z;
          } else if constexpr (FP8) {
            // their token scales too (both waves that load the scales clear
            // them after their own loads landed, so a zero is written last)
            if (wave >= 2 && (int)(lane & 31) >= valid) *(float LDS_AS*)(buf + L::kData + 4 * lane) = 0.f;
          }
        }
        if constexpr (LAT) {
          // the tile-major table of the step's scale exponents (after the
          // zero fill): (bits >> 16) - (127 << 7) is e << 7 for 2^e; a
          // zeroed scale (rows past the end, whose weights are 0) gives a
          // step that keeps those weights 0
          if (wave == 0 && lane < 32) {
            const u32x4 v = *(const u32x4 LDS_AS*)(buf + L::kData + 16 * lane);
#pragma unroll
            for (int t = 0; t < 4; ++t)
              *(uint16_t LDS_AS*)(buf + L::kScaleT + 2 * (32 * t + lane)) = (uint16_t)(((v[t] >> 16) & 0x7F80u) - 0x3F80u);
          }
        }
        // step j staged; P of step j-1 visible; every wave is done with
        // iteration j-1, so the slot of step j-2 is free
        lds_barrier();

        // ---- stream 1: QK^T of step j for the wave's head block (36 MFMAs,
        // one K fragment each) with the first kPV1 MFMAs of PV of step j-1
        // spread among them (PV MFMA q: column block c = q >> 2 of key half
        // c >> 2, head block q & 3) and the loads of step j + kDist; the other
        // 32 - kPV1 PV MFMAs run under the softmax (stream 2).
        f32x16 sacc;
        bf16x8 pf[4], pf1[4];
        u32x4 psc[2];  // LAT: tile-`wave` scale exponent steps of the keys of pf / pf1
        FragRaw<FP8> vf[3];  // V fragments of three column blocks, as read
        bf16x8 vcur;         // that of the current column block, converted
        {
          constexpr int kKPre = 4;  // K fragments in flight
          FragRaw<FP8> kf[kQ8 ? 1 : kKPre];
          // kQ8: K operands of dims blocks kb in a ring of three, each read a
          // block ahead, so a block's registers are rewritten five slots
          // (two 64-cycle MFMAs) after their last MFMA was issued
          i32x8 k8[kQ8 ? 3 : 1];
          auto load_k8 = [&](int kb) {
            const u32x2 r0 = load_k_raw<true>(buf, kbase, 4 * kb), r1 = load_k_raw<true>(buf, kbase, 4 * kb + 1);
            const u32x2 r2 = load_k_raw<true>(buf, kbase, 4 * kb + 2), r3 = load_k_raw<true>(buf, kbase, 4 * kb + 3);
            const u32x4 lo4 = __builtin_shufflevector(r0, r1, 0, 1, 2, 3), hi4 = __builtin_shufflevector(r2, r3, 0, 1, 2, 3);
            return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
          };
          bf16x8 ka_prev;  // fp8: the converted fragment the previous QK MFMA was issued with
          bf16x8 kr[4];    // LAT: the RoPE fragments, bf16 as staged
          f32x4 tsc;       // LAT: tile scales of this lane's key row
          if constexpr (LAT) tsc = *(const f32x4 LDS_AS*)(buf + L::kData + 16 * n32);
          int tsb[4];  // LAT: the tile scales' E8M0 bytes (their biased exponents)
          if constexpr (LAT) {
#pragma unroll
            for (int t = 0; t < 4; ++t) tsb[t] = (int)((__float_as_uint(tsc[t]) >> 23) & 255u);
          }
          if constexpr (kQ8) {
            k8[0] = load_k8(0);
          } else {
#pragma unroll
            for (int ks = 0; ks < kKPre; ++ks) kf[ks] = load_k_raw<FP8>(buf, kbase, ks);
          }
          if constexpr (kPV) {
            // the MFMAs step j-2 deferred, operands in registers, while the
            // first K fragments arrive
#pragma unroll
            for (int hb = 4 - kPVDefer; hb < 4; ++hb) {
              o[3][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(d_v, d_p[hb], o[3][hb], 0, 0, 0);
              __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (LAT) load_p_scales(vbuf + L::kScaleT, 0, h, wave, psc[0]);
#pragma unroll
            for (int hb = 0; hb < 4; ++hb) pf[hb] = *(const bf16x8 LDS_AS*)(p_prev + p_slot(32 * hb + n32, 0, h));
            vf[0] = load_v_raw<FP8>(vbuf, vbase, 4 * wave, 0);
            vf[1] = load_v_raw<FP8>(vbuf, vbase, 4 * wave + 1, 0);
          }
#pragma unroll
          for (int i = 0; i < 36; ++i) {
            // PV MFMA q of this slot, if any: slot (36q) / kPV1
            constexpr int kNone = -1;
            constexpr int kPV1d = kPV1 > 0 ? kPV1 : 1;  // (no division by zero when kPV1 is 0)
            const int qc = (i * kPV1 + 35) / 36;
            const int q = (kPV && qc < kPV1 && (qc * 36) / kPV1d == i) ? qc : kNone;
            if (q != kNone && (q & 3) == 0 && (q >> 2) + 2 < 8) {
              // V fragment two column blocks ahead (c = 4kh + cbl); its ring
              // entry last served column block c - 1
              const int cn = (q >> 2) + 2;
              vf[cn % 3] = load_v_raw<FP8>(vbuf, vbase, 4 * wave + (cn & 3), cn >> 2);
            }
            if constexpr (kQ8) {
              // dims block kb = i / 4: its hi MFMA in slot 4kb + 1, its lo
              // MFMA (block scale 2^-4) in slot 4kb + 3; block kb + 1 read in
              // slot 4kb.  Latent rows: K's block scale is its tile's, and the
              // bf16 RoPE fragments (read in slots 28-31) take slots 32-35.
              const int kb = i >> 2;
              if ((i & 3) == 0 && kb + 1 < kQB) k8[(kb + 1) % 3] = load_k8(kb + 1);
              if (kb < kQB) {
                const int ksc = LAT ? tsb[kb >> 1] : bs_one;
                if ((i & 3) == 1) {
                  if (kb == 0) mfma_qk8<true, LAT>(sacc, k8[kb % 3], q8[2 * kb], ksc, bs_one);
                  else mfma_qk8<false, false>(sacc, k8[kb % 3], q8[2 * kb], ksc, bs_one);
                }
                if ((i & 3) == 3) mfma_qk8<false, false>(sacc, k8[kb % 3], q8[2 * kb + 1], ksc, bs_lo);
              }
              if constexpr (LAT) {
                if (i >= 28 && i < 32) kr[i & 3] = *(const bf16x8 LDS_AS*)(buf + kbase_r[i & 3]);
                if (i >= 32) {
                  // the bf16 MFMA reads the accumulator the 16-pass fp8 MFMA
                  // wrote: its wait states first
                  if (i == 32) asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(sacc));
                  mfma_qk<false, false>(sacc, kr[i & 3], qr[i & 3]);
                }
              }
            } else {
              bf16x8 ka;
              if constexpr (LAT) ka = i < 32 ? fp8x8_scaled_to_bf16(kf[i % kKPre], tsc[i >> 3]) : kr[i & 3];
              else ka = frag_bf16<FP8>(kf[i % kKPre]);
              if constexpr (FP8) {
                // the conversion must not reuse the registers of the MFMA just
                // issued (the asm hides that read from the compiler): keeping
                // that fragment live through it gives this one its own
                if (i > 0) asm volatile("" ::"v"(ka), "v"(ka_prev));
                ka_prev = ka;
              }
              if (i + kKPre < 36) {
                if (LAT && i + kKPre >= 32) kr[(i + kKPre) & 3] = *(const bf16x8 LDS_AS*)(buf + kbase_r[(i + kKPre) & 3]);
                else kf[i % kKPre] = load_k_raw<FP8>(buf, kbase, i + kKPre);
              }
              if (i == 0) mfma_qk<true, FP8>(sacc, ka, qf[i]);
              else mfma_qk<false, FP8>(sacc, ka, qf[i]);
            }
            if (q != kNone) {
              const int c = q >> 2, hb = q & 3;
              if constexpr (LAT) {
                // P scaled at its first use (its 4 column blocks share it;
                // those of key half 1 are scaled in stream 2)
                if (c == 0) pf[hb] = scale_p(pf[hb], psc[0]);
              }
              const bf16x8 pv = c < 4 ? pf[hb] : pf1[hb];
              if (hb == 0) vcur = frag_bf16<FP8>(vf[(c + 3) % 3]);
              o[c & 3][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vcur, pv, o[c & 3][hb], 0, 0, 0);
              // key half 1 P fragment of this head block, in the registers
              // of the half 0 one, which column block 3 has just read last
              if (c == 3) pf1[hb] = *(const bf16x8 LDS_AS*)(p_prev + p_slot(32 * hb + n32, 1, h));
            }
            // the loads of step j + kDist, spread over the stream
            if ((i & 3) == 1 && (i >> 2) < L::kLoadsPerStep && pf_next) {
              if constexpr (TOPK) {
                switch (i >> 2) {
                  case 0: issue_one_v<FP8, 0, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 1: issue_one_v<FP8, 1, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 2: issue_one_v<FP8, 2, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 3: issue_one_v<FP8, 3, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 4: issue_one_v<FP8, 4, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 5: issue_one_v<FP8, 5, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 6: issue_one_v<FP8, 6, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  case 7: issue_one_v<FP8, 7, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                  default: issue_one_v<FP8, 8, LAT, NT>(pf_row, pf_srow, pf_buf, wave, pf_rows, kv); break;
                }
              } else {
                switch (i >> 2) {
                  case 0: issue_one<FP8, 0, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 1: issue_one<FP8, 1, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 2: issue_one<FP8, 2, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 3: issue_one<FP8, 3, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 4: issue_one<FP8, 4, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 5: issue_one<FP8, 5, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 6: issue_one<FP8, 6, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  case 7: issue_one<FP8, 7, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                  default: issue_one<FP8, 8, LAT, NT>(pf_src, pf_scales, src_lane, pf_buf, wave); break;
                }
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
        // PV MFMA q >= kPV1 of step j-1, with the V fragment of column block
        // c + 2 loaded at the first MFMA of column block c
        auto pv_slot = [&](int q) {
          if constexpr (kPV) {
            const int c = q >> 2, hb = q & 3;
            if (hb == 0 && c + 2 < 8) {
              const int cn = c + 2;
              vf[cn % 3] = load_v_raw<FP8>(vbuf, vbase, 4 * wave + (cn & 3), cn >> 2);
            }
            if constexpr (LAT) {
              // each P fragment is scaled at its first use (column block 0
              // or 4), here or, for the MFMAs placed there, in stream 1
              if (c == 0) pf[hb] = scale_p(pf[hb], psc[0]);
              if (c == 4) pf1[hb] = scale_p(pf1[hb], psc[1]);
            }
            const bf16x8 pv = c < 4 ? pf[hb] : pf1[hb];
            if (hb == 0) vcur = frag_bf16<FP8>(vf[c % 3]);
            if (q >= 32 - kPVDefer) {
              // carried past the next barrier
              if (hb == 4 - kPVDefer) d_v = vcur;
              d_p[hb] = pv;
            } else {
              o[c & 3][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vcur, pv, o[c & 3][hb], 0, 0, 0);
            }
            // (as in stream 1) the key half 1 P fragment after the last read
            // of the half 0 one (LAT: with its key scales)
            if (c == 3) {
              pf1[hb] = *(const bf16x8 LDS_AS*)(p_prev + p_slot(32 * hb + n32, 1, h));
              if constexpr (LAT) {
                if (hb == 0) load_p_scales(vbuf + L::kScaleT, 1, h, wave, psc[1]);
              }
            }
          }
        };
        // kLead PV MFMAs run while the QK chain drains, the last kTail after
        // the P of step j is published (through the write and the next
        // barrier); the softmax rides on the rest
        constexpr int kLead = kPV ? 2 : 0, kTail = kPV ? kPVTail + kPVDefer : 0;
        constexpr int kN2 = kPV ? 32 - kPV1 - kTail : 0;  // PV slots of stream 2
        f32x2 sc[8];
        if constexpr (FP8 && !LAT) {
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            const int m = 8 * (r >> 2) + 4 * h + (r & 3);
            sc[r >> 1] = *(const f32x2 LDS_AS*)(buf + L::kData + 4 * m);
          }
        }

        // ---- scores: token scales (fp8), the history-end mask and, on the
        // unit's first step, the reference.  Softmax in base 2; lane = one
        // head, keys 8(r>>2)+4h+(r&3); t = z*log2(e) - m_ref.
        auto finish_scores = [&]() {
          wait_mfma_vgpr(sacc);
          if constexpr (FP8 && !LAT) {
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
              sacc[r] *= sc[r >> 1][0];
              sacc[r + 1] *= sc[r >> 1][1];
            }
          }
          if (may_end && valid < kStepKeys) {
            // the last step of a history: keys past its end get no weight
            const int hk = (int)opaque(4 * h);
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (hk + (8 * (r >> 2) + (r & 3)) >= valid) sacc[r] = -INFINITY;
          }
          if constexpr (!kPV) {
            // first step of the pass: its largest score is the reference
            // (a restarted pass already has one)
            if (m_ref == -INFINITY) {
              float mx = -INFINITY;
#pragma unroll
              for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[r] * c2v);
              m_ref = fmaxf(mx, wave_xor32(mx));
            }
          }
        };
        if constexpr (!kPV) finish_scores();

        // ---- stream 2: the softmax (16 elements per lane) spread over the
        // remaining PV MFMAs of step j-1.
        // P is rounded to bf16 for the PV MFMA.  The bf16 path normalises the
        // output by the sum of the rounded weights, so the weights applied to V
        // sum to one and only the spread of the rounding errors reaches the
        // output; the LSE keeps the exact fp32 sum.
        float psum = 0.f, pexact = 0.f, plo = 0.f, tlo = 0.f;
        unsigned pb[8];
        auto softmax_elem = [&](int r) {
          const float t = __builtin_fmaf(sacc[r], c2v, -m_ref);
          const float p = __builtin_amdgcn_exp2f(t);
          pexact += p;
          if (r & 1) {
            // largest t of the pass, two per max3
            tmax = fmaxf(tmax, fmaxf(tlo, t));
            if constexpr (FP8 && !LAT) {
              // the token scale multiplies V too: fold it into the weight
              pb[r >> 1] = pack_bf16x2(plo * sc[r >> 1][0], p * sc[r >> 1][1]);
            } else {
              const unsigned w = pack_bf16x2(plo, p);
              pb[r >> 1] = w;
              psum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), (bf16x2){1.0f, 1.0f}, psum, false);
            }
          } else {
            plo = p;
            tlo = t;
          }
          // keep the element here, between the MFMAs of its slot, instead of
          // letting the compiler sink the whole softmax below the stream
          if constexpr (FP8 && !LAT) asm volatile("" : "+v"(pexact));
          else asm volatile("" : "+v"(pexact), "+v"(psum));
        };
        if constexpr (kPV) {
#pragma unroll
          for (int k = 0; k < kN2; ++k) {
            pv_slot(kPV1 + k);
            if (k == kLead - 1) finish_scores();
            // softmax elements of this slot: [ceil(16k' / S), ceil(16(k'+1) / S))
            // with k' = k - kLead over the S = N2 - kLead slots after the lead
            constexpr int kS = kN2 - kLead;
            if (k >= kLead) {
              const int kk = k - kLead;
#pragma unroll
              for (int r = (16 * kk + kS - 1) / kS; r < (16 * (kk + 1) + kS - 1) / kS; ++r) softmax_elem(r);
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r) softmax_elem(r);
        }
        l_exact += pexact;
        l_run += (FP8 && !LAT) ? pexact : psum;
        // page (top-k: rows) of the step the next iteration stages, read now
        // and used there; the index is clamped to the unit's last step.  (The
        // scalar load is issued after the last LDS wait of the iteration:
        // until it returns every LDS wait is a full one, and the next one is
        // the barrier's.)
        if (kPFM != 2) {
          const int jn = min(j + kDist + 1, nsteps - 1);
          if constexpr (TOPK) {
            next_row = lane_row(jn);
            next_srow = scale_row(jn);
          } else {
            next_phys = step_phys(jn);
          }
        }
        // publish this wave's P^T (keys in slot order) for every wave's PV
        uint8_t LDS_AS* p_cur = p_lds + kPBytes * (j & 1);
        *(u32x4 LDS_AS*)(p_cur + p_slot(head, 0, h)) = (u32x4){pb[0], pb[1], pb[2], pb[3]};
        *(u32x4 LDS_AS*)(p_cur + p_slot(head, 1, h)) = (u32x4){pb[4], pb[5], pb[6], pb[7]};
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < kTail; ++k) {
          pv_slot(kPV1 + kN2 + k);
          __builtin_amdgcn_sched_barrier(0);
        }
      };

      qk_softmax(0, std::false_type{}, std::integral_constant<int, 0>{});
      int j = 1;
      for (; j + kDist < nsteps; ++j) qk_softmax(j, std::true_type{}, std::integral_constant<int, 1>{});
      for (; j < nsteps; ++j) qk_softmax(j, std::true_type{}, std::integral_constant<int, 2>{});
      // PV of the last step
      lds_barrier();
      pv_stream<FP8, LAT>(slot_buf(nsteps - 1), vbase, p_lds + kPBytes * ((nsteps - 1) & 1), wave, n32, h, o,
                          L::kScaleT, d_v, d_p);
      const float mt_max = fmaxf(tmax, wave_xor32(tmax));
      const float m_seen = m_ref + mt_max;
      const bool over = mt_max > 64.0f;
      // Every wave votes in the P buffer the last step did not use: the last
      // PV reads only the other one.  It is written next by the P of the
      // first step of a second pass, behind that step's barrier, so every
      // wave has read the votes by then.
      int32_t LDS_AS* votes = (int32_t LDS_AS*)(p_lds + kPBytes * (nsteps & 1));
      if (lane == 0) votes[wave] = __builtin_amdgcn_ballot_w64(over) ? 1 : 0;
      __syncthreads();
      const bool restart = (votes[0] | votes[1] | votes[2] | votes[3]) != 0;
      // the second pass starts from the unit's true max, so it never
      // overflows; it is the last one in any case
      if (!restart || pass > 0) break;
      m_init = m_seen;
    }  // pass

    // ---- the next unit's query and first steps.  Every wave is past its
    // last PV (the vote barrier), so the ring is free; the epilogue below
    // stages in LDS these steps do not use.  Steps 0 and 1 are the two halves
    // of the unit's first page.
    pre = false;
    if constexpr (kOverlap) {
      if (nxt.x >= 0) {
        load_q(N.tile);
#pragma unroll
        for (int j = 0; j < kDist; ++j)
          if (j < N.nsteps) issue_step<FP8, LAT, NT>(step_src(j, n_phys), step_scales(j, n_phys), src_lane, slot_buf(j), wave);
        pre = true;
      }
    }

    // ---- epilogue: normalise and store
    {
      // normaliser: sum of the weights as applied (rounded); LSE: exact sum
      const float l_tot = l_run + wave_xor32(l_run);
      const float l_ex = l_exact + wave_xor32(l_exact);
      const float lse_nat = (m_ref + __log2f(l_ex)) * 0.6931471805599453f;
      // the reciprocal of each head's normaliser (1 ulp), by the wave that
      // owns the head, at 32 hb + 16 (head & 1) + (head & 31) / 2: the
      // store lanes below find their 16 rows of a head block contiguous
      if (h == 0) l_lds[(head & ~31) + 16 * (head & 1) + ((head & 31) >> 1)] = __builtin_amdgcn_rcpf(l_tot);
      if (h == 0 && head_ok) {
        if (slot < 0) {
          if (a.lse) a.lse[(size_t)tile * a.H + head] = lse_nat;
        } else {
          a.ws.part_lse[(size_t)slot * a.H + head] = lse_nat;
        }
      }
    }
    __syncthreads();
    // Each head block goes through LDS (the ring is free: every wave is past
    // its last PV and no load is in flight), so that the stores write whole
    // rows (256 B of fp16 or bf16 per head) instead of the
    // accumulators' 32-byte pieces spread over 32 rows.  NT: the stores are
    // non-temporal too.  Lines left dirty in the L2 are written back at the
    // kernel's end, after the last worker; streamed stores shorten that
    // drain, at the price of the combine reading the partials from memory
    // instead of the L2 (measured on the one-row-per-request workloads: the
    // kernel 2-7 us shorter, the combine 2 us longer).  Each wave stages its
    // own 128 columns; its LDS ops complete in order, so no barrier is needed.
    // Accumulator lane: head 32hb + n32, columns 32cbl + 8q + 4h + [0, 4).
    {
      // The addresses below are the same for every unit: laundering the lane
      // coordinates here keeps the compiler from hoisting all of them out of
      // the unit loop (and spilling them).
      const int hl = (int)opaque((uint32_t)h), nl = (int)opaque((uint32_t)n32);
      const uint8_t LDS_AS* wstage = sm + kStageOff + wave * 32 * kStageRow;
      auto rows = [&](int hb, auto store) {
        // rows 2k + h, 4 columns per lane: 32 lanes cover one head's 128,
        // scaled by the row's reciprocal normaliser.  Rows go in batches of
        // eight: their reads are issued together (the empty asm keeps them
        // ahead of the stores), then their stores.  Heads past H are not
        // stored: as H is a multiple of 16, the rows of head block hb to
        // store are k < (H - 32 hb) / 2, a multiple of 8, the same for the
        // whole wave.
        // (a split partial: this wave's normalisers, times each quarter's scale)
        const float LDS_AS* l_rows =
            slot >= 0 ? (const float LDS_AS*)(sm + kStageOff + kScOff) + kMaxHeads * wave : l_lds;
        f32x4 rl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) rl[i] = *(const f32x4 LDS_AS*)(l_rows + 32 * hb + 16 * hl + 4 * i);
        const int kval = min(16, (a.H - 32 * hb) / 2);
#pragma unroll 1
        for (int k0 = 0; k0 < kval; k0 += 8) {
          f32x4 v[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) v[k] = *(const f32x4 LDS_AS*)(wstage + (2 * (k0 + k) + hl) * kStageRow + nl * 16);
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const f32x4 r = k0 ? rl[2 + (k >> 2)] : rl[k >> 2];
            v[k] *= r[k & 3];
            asm volatile("" : "+v"(v[k]));
          }
#pragma unroll
          for (int k = 0; k < 8; ++k) store(32 * hb + 2 * (k0 + k) + hl, v[k]);
        }
      };
      const size_t col = 128 * wave + 4 * nl;
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
        uint8_t LDS_AS* stage = sm + kStageOff + wave * 32 * kStageRow + nl * kStageRow + 16 * hl;
#pragma unroll
        for (int cbl = 0; cbl < 4; ++cbl)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *(f32x4 LDS_AS*)(stage + (32 * cbl + 8 * q) * 4) =
                (f32x4){o[cbl][hb][4 * q], o[cbl][hb][4 * q + 1], o[cbl][hb][4 * q + 2], o[cbl][hb][4 * q + 3]};
        if (slot >= 0) {
          // split partial: the largest magnitude of the lane's 64 columns,
          // read back from the staged copy (through a laundered address, so
          // that the compiler does not keep the accumulator values for it)
          const uint8_t LDS_AS* rb =
              sm + opaque((uint32_t)(kStageOff + wave * 32 * kStageRow + nl * kStageRow + 16 * hl));
          float m = 0.f;
#pragma unroll
          for (int cbl = 0; cbl < 4; ++cbl)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const f32x4 x = *(const f32x4 LDS_AS*)(rb + (32 * cbl + 8 * q) * 4);
              m = fmaxf(m, fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3]))));
            }
          // the quarter's scale: lanes n32 and n32 + 32 hold head 32 hb + n32's
          // 128 columns of this wave; the scale goes to this wave's table at
          // the normaliser's index (read back below by the lanes that store
          // the head's rows), its exponent to byte `wave` of the head's word
          m = fmaxf(m, wave_xor32(m));
          const int li = 32 * hb + 16 * (nl & 1) + (nl >> 1);
          const float rcp = l_lds[li];
          const uint32_t e = partial_exponent(m * rcp);
          if (hl == 0) {
            ((float LDS_AS*)(sm + kStageOff + kScOff))[kMaxHeads * wave + li] = rcp * __builtin_bit_cast(float, (127u - e) << 23);
            if (32 * hb + nl < a.H) ((uint8_t*)(a.ws.part_exp + (size_t)slot * a.H + 32 * hb + nl))[wave] = (uint8_t)e;
          }
        }
        if (slot < 0) {
          uint16_t* obase = (uint16_t*)a.out + (size_t)tile * a.H * kDimV + col;
          rows(hb, [&](int hh, const f32x4& v) {
            u32x2 w;
            w[0] = pack_bf16x2(v[0], v[1]);
            w[1] = pack_bf16x2(v[2], v[3]);
            if constexpr (NT) __builtin_nontemporal_store(w, (u32x2*)(obase + (size_t)hh * kDimV));
            else *(u32x2*)(obase + (size_t)hh * kDimV) = w;
          });
        } else {
          uint16_t* pbase = a.ws.part_half + (size_t)slot * a.H * kDimV + col;
          rows(hb, [&](int hh, const f32x4& v) {
            u32x2 w;
            w[0] = pack_f16x2(v[0], v[1]);
            w[1] = pack_f16x2(v[2], v[3]);
            if constexpr (NT) __builtin_nontemporal_store(w, (u32x2*)(pbase + (size_t)hh * kDimV));
            else *(u32x2*)(pbase + (size_t)hh * kDimV) = w;
          });
        }
      }
    }
    cur = nxt;
    nxt = nxt2;
  }
}

// ============================================================== combine ===

constexpr int kCombineQuarters = 4;  // waves per (row, head): 128 columns each
constexpr int kCombineRowParts = 8;  // at most this many parts: one wave per (row, head)
//
// The standalone merge of fp32 partials by split offsets (splash_mla_combine).
// Four wave slots per (request, chunk row, head), 128 columns each (2 per
// lane).  With at most 8 parts every lane loads all parts' LSEs and its
// columns of all parts at once; with more, the LSEs are reduced across the
// lanes first and sixteen parts' columns are in flight at a time.
__global__ __launch_bounds__(256) void combine_kernel(CombineLaunch c) {
  const int lane = threadIdx.x & 63;
  const int64_t wave_global = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  if (c.B <= 0) return;
  const size_t stride = (size_t)c.q_chunk * c.H;  // between parts
  // output row of (item b, chunk row qi): b * q_chunk + qi, or its place
  // among the shards
  auto out_row = [&](int b, int qi) -> size_t {
    const size_t r = (size_t)b * c.q_chunk + qi;
    if (c.num_shards <= 0) return r;
    const size_t rb = r / (size_t)c.tile_q, ri = r - rb * (size_t)c.tile_q;
    return (rb * c.num_shards + c.shard) * c.tile_q + ri;
  };
  // One wave per (item, row, head) with at most kCombineRowParts parts: 8
  // columns per lane, every part's LSE and columns loaded at once, so the row
  // costs one round trip to memory for its data and no cross-lane reduction.
  auto row_merge = [&](int b, int s0, int np, int qi, int hh) {
    const size_t base = (size_t)qi * c.H + hh;
    const size_t orow = out_row(b, qi) * c.H + hh;
    const float* plse = c.partial_lse + base;
    f32x4 v[kCombineRowParts][2];
    float w[kCombineRowParts];
    const float* prow = c.partials + base * kDimV + 8 * lane;
#pragma unroll
    for (int u = 0; u < kCombineRowParts; ++u) {
      w[u] = -INFINITY;
      v[u][0] = v[u][1] = (f32x4){0.f, 0.f, 0.f, 0.f};
      if (u < np) {  // uniform
        w[u] = plse[(size_t)(s0 + u) * stride];
        const f32x4* src = (const f32x4*)(prow + (size_t)(s0 + u) * stride * kDimV);
        v[u][0] = src[0];
        v[u][1] = src[1];
      }
    }
    float M = -INFINITY, wsum = 0.f;
#pragma unroll
    for (int u = 0; u < kCombineRowParts; ++u) M = fmaxf(M, w[u]);
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    if (M > -INFINITY) {
#pragma unroll
      for (int u = 0; u < kCombineRowParts; ++u) {
        const float wu = __expf(w[u] - M);  // 0 past the last part
        wsum += wu;
        acc0 += wu * v[u][0];
        acc1 += wu * v[u][1];
      }
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    if (c.out_f32) {
      f32x4* dst = (f32x4*)((float*)c.out + orow * kDimV + 8 * lane);
      dst[0] = acc0 * inv;
      dst[1] = acc1 * inv;
    } else {
      u32x4 o4;
      o4[0] = pack_bf16x2(acc0[0] * inv, acc0[1] * inv);
      o4[1] = pack_bf16x2(acc0[2] * inv, acc0[3] * inv);
      o4[2] = pack_bf16x2(acc1[0] * inv, acc1[1] * inv);
      o4[3] = pack_bf16x2(acc1[2] * inv, acc1[3] * inv);
      *(u32x4*)((uint16_t*)c.out + orow * kDimV + 8 * lane) = o4;
    }
    if (lane == 0 && c.out_lse) c.out_lse[orow] = wsum > 0.f ? M + __logf(wsum) : -INFINITY;
  };
  // one (request or tile, row, head, quarter) item
  auto combine_item = [&](int b, int s0, int s1, int quarter, int qi, int hh) {
    const size_t orow = out_row(b, qi) * c.H + hh;
    const int nparts = s1 - s0;
    const size_t base = (size_t)qi * c.H + hh;
    const float* plse = c.partial_lse + base;
    const int col = 128 * quarter + 2 * lane;
    // the lane's 2 columns of part s (fp32 partials: this path serves the
    // standalone merge)
    auto part2 = [&](int sp) -> f32x2 { return *(const f32x2*)(c.partials + ((size_t)sp * stride + base) * kDimV + col); };
    float M = -INFINITY, wsum = 0.f;
    f32x2 acc = {0.f, 0.f};
    if (nparts <= 8) {
      // few parts: every lane loads every part's LSE itself (the same 32
      // bytes for the whole wave) together with its 2 columns of every part,
      // so the row costs one round trip to memory and no cross-lane reduction
      f32x2 v[8];
      float w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        w[u] = -INFINITY;
        v[u] = (f32x2){0.f, 0.f};
        if (u < nparts) {  // uniform
          w[u] = plse[(size_t)(s0 + u) * stride];
          v[u] = part2(s0 + u);
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) M = fmaxf(M, w[u]);
      if (M > -INFINITY) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float wu = __expf(w[u] - M);  // 0 past the last part
          wsum += wu;
          acc += wu * v[u];
        }
      }
    } else {
      for (int s = s0 + lane; s < s1; s += 64) M = fmaxf(M, plse[(size_t)s * stride]);
      M = __ockl_wfred_max_f32(M);
      if (M > -INFINITY)
        for (int s = s0 + lane; s < s1; s += 64) wsum += __expf(plse[(size_t)s * stride] - M);
      wsum = __ockl_wfred_add_f32(wsum);
      // many parts: sixteen parts' columns in flight at a time
      if (M > -INFINITY) {
        constexpr int kU = 16;
        int s = s0;
        for (; s + kU <= s1; s += kU) {
          f32x2 v[kU];
          float w[kU];
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            v[u] = part2(s + u);
            w[u] = plse[(size_t)(s + u) * stride];
          }
#pragma unroll
          for (int u = 0; u < kU; ++u) acc += __expf(w[u] - M) * v[u];
        }
        if (s < s1) {
          // the remaining parts: independent loads, clamped to a valid part
          f32x2 v[kU];
          float w[kU];
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            const int su = s + u < s1 ? s + u : s1 - 1;
            v[u] = part2(su);
            w[u] = s + u < s1 ? plse[(size_t)su * stride] : -INFINITY;
          }
#pragma unroll
          for (int u = 0; u < kU; ++u) acc += __expf(w[u] - M) * v[u];
        }
      }
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    if (c.out_f32)
      *(f32x2*)((float*)c.out + orow * kDimV + col) = acc * inv;
    else
      *(unsigned*)((uint16_t*)c.out + orow * kDimV + col) = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    if (lane == 0 && quarter == 0 && c.out_lse) c.out_lse[orow] = wsum > 0.f ? M + __logf(wsum) : -INFINITY;
  };
  {
    // one wave per (request, row, head), which takes the one-round-trip row
    // merge when the request has at most kCombineRowParts parts and
    // otherwise the four quarters in turn
    const int64_t per_b = (int64_t)c.q_chunk * c.H;
    for (int64_t item = wave_global; item < (int64_t)c.B * per_b; item += nwaves) {
      const int b = (int)(item / per_b);
      const int row = (int)(item - (int64_t)b * per_b);
      const int qi = row / c.H, hh = row - qi * c.H;
      const int s0 = c.indptr[b], s1 = c.indptr[b + 1];
      if (s1 <= s0 && !c.write_empty) continue;
      if (s1 - s0 <= kCombineRowParts) {
        row_merge(b, s0, s1 - s0, qi, hh);
      } else {
        for (int quarter = 0; quarter < kCombineQuarters; ++quarter) combine_item(b, s0, s1, quarter, qi, hh);
      }
    }
  }
}

// The merge of one step's split partials (splash_mla_combine_splits): the
// attend kernel's fp16 partials with their quarter exponents, the split
// tiles listed by the planner.  Every (tile, chunk row, head) row is one
// item; a lane holds 8 of its 512 columns (quarter lane / 16).  With at most
// kMergeWaveParts parts per tile (the plan's bound), or with at least
// kMergeWaveItems items of at most kMergeWaveLongParts parts (items enough
// to fill the chip with waves, so a workgroup per item would only queue
// them), a wave takes an item alone; otherwise a workgroup takes it and its
// four waves split the parts.  Either way parts go kMergeBatch at a time,
// one memory round trip per batch, against a running maximum of their LSEs
// (the sums rescaled when it grows); the four waves of a workgroup meet in
// LDS.  Few registers, so that many waves hide the round trips.
constexpr int kMergeWaveParts = 4;
constexpr int kMergeWaveItems = 8192;
constexpr int kMergeWaveLongParts = 16;
constexpr int kMergeBatch = 4;
__global__ __launch_bounds__(256) void merge_splits_kernel(CombineLaunch c) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t nitems = (int64_t)(*c.item_count) * c.q_chunk * c.H;
  if (nitems == 0) return;
  const int max_parts = *c.max_parts;
  const bool by_wave = max_parts <= kMergeWaveParts ||
                       (nitems >= kMergeWaveItems && max_parts <= kMergeWaveLongParts);  // uniform
  const size_t stride = (size_t)c.q_chunk * c.H;          // between parts
  const int qsh = 8 * (lane >> 4);
  // parts first, first + step, ... of an item: running max m, weight sum,
  // column sums
  auto accumulate = [&](const int4& rec, size_t base, int first, int step, float& m, float& ssum, f32x4& acc0,
                        f32x4& acc1) {
    const int s0 = rec.y, np = rec.z;
    const float* plse = c.partial_lse + base;
    const uint16_t* prow = c.partials_h + base * kDimV + 8 * lane;
    for (int u0 = first; u0 < np; u0 += step * kMergeBatch) {
      u32x4 raw[kMergeBatch];
      float wu[kMergeBatch];
      uint32_t ew[kMergeBatch];
#pragma unroll
      for (int k = 0; k < kMergeBatch; ++k) {
        const int u = u0 + step * k;
        raw[k] = (u32x4){0, 0, 0, 0};
        wu[k] = -INFINITY;
        ew[k] = 0;
        if (u < np) {  // uniform
          const size_t r = (size_t)(s0 + u) * stride;
          raw[k] = *(const u32x4*)(prow + r * kDimV);
          wu[k] = plse[r];
          ew[k] = c.part_exp[r + base];
        }
      }
      float bm = -INFINITY;
#pragma unroll
      for (int k = 0; k < kMergeBatch; ++k) bm = fmaxf(bm, wu[k]);
      if (bm > -INFINITY) {  // uniform
        const float mn = fmaxf(m, bm), rs = __expf(m - mn);  // 0 while m is -inf
        acc0 *= rs;
        acc1 *= rs;
        ssum *= rs;
        m = mn;
#pragma unroll
        for (int k = 0; k < kMergeBatch; ++k) {
          const int e = (int)((ew[k] >> qsh) & 255u);
          const float sc = __expf(wu[k] - m);  // 0 for parts past the end
          ssum += sc;
          acc0 += sc * unpack_f16x4(raw[k][0], raw[k][1], e);
          acc1 += sc * unpack_f16x4(raw[k][2], raw[k][3], e);
        }
      }
    }
  };
  auto store = [&](const int4& rec, int qi, int hh, float M, float wsum, const f32x4& acc0, const f32x4& acc1) {
    size_t r = (size_t)rec.x * c.q_chunk + qi;
    if (c.num_shards > 0) {
      const size_t rb = r / (size_t)c.tile_q, ri = r - rb * (size_t)c.tile_q;
      r = (rb * c.num_shards + c.shard) * c.tile_q + ri;
    }
    const size_t orow = r * c.H + hh;
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    if (c.out_f32) {
      f32x4* dst = (f32x4*)((float*)c.out + orow * kDimV + 8 * lane);
      dst[0] = acc0 * inv;
      dst[1] = acc1 * inv;
    } else {
      u32x4 o4;
      o4[0] = pack_bf16x2(acc0[0] * inv, acc0[1] * inv);
      o4[1] = pack_bf16x2(acc0[2] * inv, acc0[3] * inv);
      o4[2] = pack_bf16x2(acc1[0] * inv, acc1[1] * inv);
      o4[3] = pack_bf16x2(acc1[2] * inv, acc1[3] * inv);
      *(u32x4*)((uint16_t*)c.out + orow * kDimV + 8 * lane) = o4;
    }
    if (lane == 0 && c.out_lse) c.out_lse[orow] = wsum > 0.f ? M + __logf(wsum) : -INFINITY;
  };
  const int64_t per_tile = (int64_t)c.q_chunk * c.H;
  if (by_wave) {
    const int64_t nwaves = (int64_t)gridDim.x * 4;
    for (int64_t item = (int64_t)blockIdx.x * 4 + w; item < nitems; item += nwaves) {
      const int64_t ri = item / per_tile;
      const int row = (int)(item - ri * per_tile), qi = row / c.H, hh = row - qi * c.H;
      const int4 rec = c.item_list[ri];
      float m = -INFINITY, ssum = 0.f;
      f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
      accumulate(rec, (size_t)qi * c.H + hh, 0, 1, m, ssum, acc0, acc1);
      store(rec, qi, hh, m, ssum, acc0, acc1);
    }
    return;
  }
  __shared__ f32x4 s_acc[4][64][2];
  __shared__ float s_ms[4][2];
  for (int64_t item = blockIdx.x; item < nitems; item += gridDim.x) {
    const int64_t ri = item / per_tile;
    const int row = (int)(item - ri * per_tile), qi = row / c.H, hh = row - qi * c.H;
    const int4 rec = c.item_list[ri];
    float m = -INFINITY, ssum = 0.f;
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    accumulate(rec, (size_t)qi * c.H + hh, w, 4, m, ssum, acc0, acc1);
    s_acc[w][lane][0] = acc0;
    s_acc[w][lane][1] = acc1;
    if (lane == 0) {
      s_ms[w][0] = m;
      s_ms[w][1] = ssum;
    }
    __syncthreads();
    if (w == 0) {
      float M = -INFINITY;
#pragma unroll
      for (int v = 0; v < 4; ++v) M = fmaxf(M, s_ms[v][0]);
      float wsum = 0.f;
      acc0 = acc1 = (f32x4){0.f, 0.f, 0.f, 0.f};
      if (M > -INFINITY) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float f = __expf(s_ms[v][0] - M);  // 0 for a wave without parts
          wsum += f * s_ms[v][1];
          acc0 += f * s_acc[v][lane][0];
          acc1 += f * s_acc[v][lane][1];
        }
      }
      store(rec, qi, hh, M, wsum, acc0, acc1);
    }
    __syncthreads();  // s_acc and s_ms are free for the next item
  }
}

// =============================================================== gather ===
//
// Dense copy of every history through the page-address arithmetic of the
// attend kernel: token j of request b is row (block_table[b][j>>6] << 6) |
// (j & 63).  One block per request; 16-byte copies.
__global__ __launch_bounds__(256) void gather_kernel(const uint8_t* kv, const int32_t* bt, const int32_t* seq_lens,
                                                     int32_t B, int32_t bt_stride, int32_t row_bytes,
                                                     uint8_t* dense) {
  const int b = blockIdx.x;
  size_t off = 0;
  for (int r = 0; r < b; ++r) off += (size_t)seq_lens[r];
  const int s = seq_lens[b];
  const int chunks = row_bytes / 16;
  for (int64_t e = threadIdx.x; e < (int64_t)s * chunks; e += blockDim.x) {
    const int j = (int)(e / chunks), ch = (int)(e - (int64_t)j * chunks);
    const int phys = bt[(size_t)b * bt_stride + (j >> 6)];
    const uint8_t* src = kv + ((size_t)phys * kPage + (j & 63)) * row_bytes + ch * 16;
    *(u32x4*)(dense + (off + j) * row_bytes + ch * 16) = *(const u32x4*)src;
  }
}

// ================================================================ check ===
//
// Validates device data: q_chunk <= seq_lens[b] and every used block-table
// entry in [0, num_pages); under a shard also 0 <= key_begin[b] <= key_end[b]
// with key_begin[b] a page boundary, and only the shard's pages are used.
// Writes the smallest failing request + 1 (or 0).
// latent_kv (the fp8 latent-row pool, else null): once every page entry of a
// request is in range, each of its rows' four tile scales must be a positive
// normal power of two no larger than 2^63.
__global__ __launch_bounds__(256) void check_kernel(const int32_t* bt, const int32_t* seq_lens,
                                                    const int32_t* key_begin, const int32_t* key_end, int32_t B,
                                                    int32_t q_chunk, int32_t bt_stride, int32_t num_pages,
                                                    const uint8_t* latent_kv, int32_t* result) {
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    const int s = seq_lens[b];
    bool bad = s < q_chunk || (int64_t)(s + kPage - 1) / kPage > bt_stride;
    int lo = 0, hi = s;
    if (key_end) {
      lo = key_begin[b];
      hi = min(s, key_end[b]);
      bad = bad || lo < 0 || (lo & (kPage - 1)) != 0 || key_end[b] < lo;
    }
    if (!bad && hi > lo) {
      const int np = (hi + kPage - 1) / kPage;
      for (int k = lo / kPage + threadIdx.x; k < np; k += blockDim.x) {
        const int v = bt[(size_t)b * bt_stride + k];
        if (v < 0 || v >= num_pages) bad = true;
      }
    }
    if (latent_kv && !__syncthreads_or(bad) && hi > lo) {
      for (int j = lo + threadIdx.x; j < hi; j += blockDim.x) {
        const size_t row = (size_t)bt[(size_t)b * bt_stride + (j >> 6)] * kPage + (j & (kPage - 1));
        const u32x4 sc = *(const u32x4*)(latent_kv + row * kLatentRowBytes + 512);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint32_t e = (sc[t] >> 23) & 0xFF;
          if ((sc[t] & 0x807FFFFFu) != 0 || e == 0 || e > 127 + 63) bad = true;
        }
      }
    }
    if (bad) atomicMin(result, b + 1);
  }
}

__global__ void init_check(int32_t* result) { *result = INT32_MAX; }

// Top-k variant: every row's count in [0, topk], every used position in the
// row's visible prefix [0, s_b - q_chunk + i], and its page's block-table
// entry in [0, num_pages); with the fp8 latent-row pool (latent_kv non-null)
// also each listed row's four tile scales a positive normal power of two
// no larger than 2^63.
// Writes the smallest failing row + 1 (or 0).
__global__ __launch_bounds__(256) void topk_check_kernel(const int32_t* bt, const int32_t* seq_lens,
                                                         const int32_t* idx, const int32_t* count, int32_t N,
                                                         int32_t q_chunk, int32_t topk, int32_t bt_stride,
                                                         int32_t num_pages, const uint8_t* latent_kv,
                                                         int32_t* result) {
  for (int n = blockIdx.x; n < N; n += gridDim.x) {
    const int b = n / q_chunk, i = n - b * q_chunk;
    const int s = seq_lens[b], c = count[n];
    const int vis = s - q_chunk + i + 1;
    bool bad = s < q_chunk || (int64_t)(s + kPage - 1) / kPage > bt_stride || c < 0 || c > topk;
    if (!bad) {
      for (int e = threadIdx.x; e < c; e += blockDim.x) {
        const int pos = idx[(size_t)n * topk + e];
        if (pos < 0 || pos >= vis) {
          bad = true;
        } else {
          const int pg = bt[(size_t)b * bt_stride + (pos >> 6)];
          if (pg < 0 || pg >= num_pages) {
            bad = true;
          } else if (latent_kv) {
            const size_t row = (size_t)pg * kPage + (pos & (kPage - 1));
            const u32x4 sc = *(const u32x4*)(latent_kv + row * kLatentRowBytes + 512);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const uint32_t ex = (sc[t] >> 23) & 0xFF;
              if ((sc[t] & 0x807FFFFFu) != 0 || ex == 0 || ex > 127 + 63) bad = true;
            }
          }
        }
      }
    }
    if (bad) atomicMin(result, n + 1);
  }
}

// ============================================================ launchers ===

hipError_t launch_plan(const PlanLaunch& p, hipStream_t s) {
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, p);
  return hipGetLastError();
}

// NT (non-temporal cache-row loads) when every request has one query row:
// then no two tiles read the same pages.
template <bool FP8, bool TOPK, bool LAT, bool Q8>
static void launch_attend_nt(const AttendLaunch& a, int32_t workers, hipStream_t s) {
  if (a.q_chunk == 1)
    hipLaunchKernelGGL((attend_kernel<FP8, TOPK, LAT, true, Q8>), dim3(workers), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attend_kernel<FP8, TOPK, LAT, false, Q8>), dim3(workers), dim3(256), 0, s, a);
}
// fp8 caches: QK on the fp8 pipe unless the caller asked for the exact one
template <bool TOPK, bool LAT>
static void launch_attend_fp8(const AttendLaunch& a, int32_t workers, hipStream_t s) {
  if (a.exact_qk) launch_attend_nt<true, TOPK, LAT, false>(a, workers, s);
  else launch_attend_nt<true, TOPK, LAT, true>(a, workers, s);
}

hipError_t launch_attend(const AttendLaunch& a, int32_t workers, hipStream_t s) {
  if (a.kv_dtype == 2) {
    if (a.topk_idx) launch_attend_fp8<true, true>(a, workers, s);
    else launch_attend_fp8<false, true>(a, workers, s);
  } else if (a.kv_dtype == 1) {
    if (a.topk_idx) launch_attend_fp8<true, false>(a, workers, s);
    else launch_attend_fp8<false, false>(a, workers, s);
  } else {
    if (a.topk_idx) launch_attend_nt<false, true, false, false>(a, workers, s);
    else launch_attend_nt<false, false, false, false>(a, workers, s);
  }
  return hipGetLastError();
}

hipError_t launch_combine(const CombineLaunch& c, hipStream_t s) {
  if (c.item_list) {
    // the step's split tiles (their number is on the device): a block per
    // (tile, row, head) up to the bound, the kernel strides over the rest
    int64_t blocks = (int64_t)c.B * c.q_chunk * c.H;
    if (blocks > 8192) blocks = 8192;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(merge_splits_kernel, dim3((unsigned)blocks), dim3(256), 0, s, c);
    return hipGetLastError();
  }
  int64_t items = (int64_t)c.B * c.q_chunk * c.H * kCombineQuarters;
  int64_t blocks = (items + 3) / 4;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)blocks), dim3(256), 0, s, c);
  return hipGetLastError();
}

hipError_t launch_gather(const void* kv, const int32_t* bt, const int32_t* seq_lens, int32_t B, int32_t bt_stride,
                         int32_t row_bytes, void* dense, hipStream_t s) {
  hipLaunchKernelGGL(gather_kernel, dim3(B), dim3(256), 0, s, (const uint8_t*)kv, bt, seq_lens, B, bt_stride,
                     row_bytes, (uint8_t*)dense);
  return hipGetLastError();
}

hipError_t launch_topk_check(const int32_t* bt, const int32_t* seq_lens, const int32_t* idx, const int32_t* count,
                             int32_t N, int32_t q_chunk, int32_t topk, int32_t bt_stride, int32_t num_pages,
                             const void* latent_kv, int32_t* result, hipStream_t s) {
  hipLaunchKernelGGL(init_check, dim3(1), dim3(1), 0, s, result);
  int blocks = N < 1024 ? N : 1024;
  hipLaunchKernelGGL(topk_check_kernel, dim3(blocks), dim3(256), 0, s, bt, seq_lens, idx, count, N, q_chunk, topk,
                     bt_stride, num_pages, (const uint8_t*)latent_kv, result);
  return hipGetLastError();
}

hipError_t launch_check(const int32_t* bt, const int32_t* seq_lens, const void* latent_kv, const int32_t* key_begin,
                        const int32_t* key_end, int32_t B, int32_t q_chunk, int32_t bt_stride, int32_t num_pages,
                        int32_t* result, hipStream_t s) {
  hipLaunchKernelGGL(init_check, dim3(1), dim3(1), 0, s, result);
  int blocks = B < 1024 ? B : 1024;
  hipLaunchKernelGGL(check_kernel, dim3(blocks), dim3(256), 0, s, bt, seq_lens, key_begin, key_end, B, q_chunk,
                     bt_stride, num_pages, (const uint8_t*)latent_kv, result);
  return hipGetLastError();
}

}  // namespace splash
