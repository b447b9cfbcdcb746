// Shared constants, parameter blocks and the single-source split planner.
//
// Everything here compiles for the host (the C-ABI validation and the host
// mirror of the planner) and for gfx950 (the kernels).
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define SPLASH_HD __host__ __device__ __forceinline__
#else
#define SPLASH_HD inline
#endif

namespace splash {

constexpr int kPage = 64;          // tokens per page
constexpr int kDimQK = 576;        // latent 512 + rope 64 (d_q = d_c + d_r)
constexpr int kDimV = 512;         // d_z = d_c
constexpr int kMaxHeads = 128;
constexpr int kStepKeys = 32;      // keys per pipeline step (half a page)
constexpr int kMaxUnitPages = 1024;  // the block-table slice of one unit is staged in LDS
constexpr int kHeaderInts = 64;

// ---------------------------------------------------------------- planner --
//
// A tile is one query row n = b*q_chunk + i with all H heads; it sees
// L = s_b - q_chunk + i + 1 keys (its complete causal prefix), i.e.
// ceil(L/64) pages.  The planner cuts each tile's page range into units of at
// most c pages; a tile cut into more than one unit writes fp32 partials that
// the combine step merges.  c is chosen by an argmin of an estimated
// makespan over candidate sizes: the units of all tiles are list-scheduled
// on G persistent workers, so the estimate is the mean load plus half the
// largest unit, with a fixed cost per unit (query load, pipeline fill) and
// per split unit (partial write + read back), in page equivalents.

struct PlanCosts {
  int32_t unit_x16;   // per-unit overhead, pages * 16
  int32_t split_x16;  // extra per unit of a split tile, pages * 16
};

constexpr PlanCosts kPlanCosts = {40, 56};
constexpr int kNumCandidates = 96;

SPLASH_HD int32_t tile_keys(int32_t seq_len, int32_t q_chunk, int32_t i) {
  return seq_len - q_chunk + i + 1;
}

SPLASH_HD int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

// Candidate unit size k (0-based): ceil(maxP / (k+1)) for k < 64, then a
// geometric continuation so very long tiles can be cut finely.
SPLASH_HD int32_t plan_candidate(int32_t k, int32_t max_pages) {
  int32_t parts = k + 1;
  if (k >= 64) {
    parts = 64;
    for (int32_t j = 64; j <= k; ++j) parts += parts / 8;
  }
  int32_t c = ceil_div(max_pages, parts);
  if (c > kMaxUnitPages) c = kMaxUnitPages;
  return c < 1 ? 1 : c;
}

// Estimated makespan (page equivalents * 16) of unit size c, given the
// number of units W and split units S it produces.
SPLASH_HD int64_t plan_cost(int32_t c, int64_t W, int64_t S, int64_t total_pages,
                            int32_t max_pages, int32_t G, PlanCosts k) {
  int64_t work = total_pages * 16 + (int64_t)k.unit_x16 * W + (int64_t)k.split_x16 * S;
  int32_t biggest = c < max_pages ? c : max_pages;
  int64_t big = (int64_t)biggest * 16 + k.unit_x16 + (c < max_pages ? k.split_x16 : 0);
  return work / G + big / 2;
}

// Unit u (0-based) of a tile of P pages cut into n units: [P*u/n, P*(u+1)/n).
SPLASH_HD int32_t unit_begin(int32_t P, int32_t n, int32_t u) {
  return (int32_t)(((int64_t)P * u) / n);
}

// ------------------------------------------------------------- LDS layout --
//
// A step stages 32 cache rows in LDS.  Rows keep their 16-byte chunks but the
// chunk order inside each aligned group of 8 (bf16) or 4 (fp8) chunks is
// XOR-permuted by row, so that the MFMA operand reads of 32 consecutive rows
// spread over the LDS banks.
SPLASH_HD uint32_t swz_bf16(uint32_t row) {
  uint32_t g = ((row & 3u) << 1) | ((row >> 2) & 1u);
  return g ^ (((row >> 3) & 1u) << 1);
}
SPLASH_HD uint32_t swz_fp8(uint32_t row) { return (row >> 1) & 3u; }

}  // namespace splash
