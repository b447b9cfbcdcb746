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
constexpr int kLatentRowBytes = 656;  // fp8 latent-row cache: 512 E4M3 + 4 fp32 tile scales + 64 bf16 RoPE
constexpr int kMaxHeads = 128;
constexpr int kStepKeys = 32;      // keys per pipeline step (half a page)
constexpr int kMaxUnitPages = 1024;  // the largest unit: the planner's length histograms and fold caps count to it
constexpr int kTopkUnitPages = 32;   // top-k variant: a unit holds 32 x 64 selected rows' addresses in LDS
constexpr int kMaxWorkers = 1024;    // the fold plan's per-worker table is sized for this many
constexpr int kHeaderInts = 1152;    // 64 header slots, then the per-worker table (kMaxWorkers + 1)
constexpr int kPlanLdsTiles = 8192;  // planner: tile data cached in LDS, and the unit queue ordered longest
                                     // first, up to this many tiles

// ---------------------------------------------------------------- planner --
//
// A tile is one query row n = b*q_chunk + i with all H heads; it sees
// L = s_b - q_chunk + i + 1 keys (its complete causal prefix), i.e.
// ceil(L/64) pages.  The planner cuts each tile's page range into units of at
// most c pages; a tile cut into more than one unit writes partials that
// the combine step merges.  c is chosen by an argmin of an estimated step
// time over candidate sizes.  The G persistent workers are dealt the units of
// a queue, so with W units the busiest worker runs R = ceil(W / G) of them: the
// estimate is max(R * c, work / G) plus, per unit on that worker, a fixed
// cost (query load, pipeline fill), per split unit on it the partial write,
// and the combine's read of all S partials spread over the workers; all in
// page equivalents, scaled by 16 G so the arithmetic is integral.

struct PlanCosts {
  int32_t unit_x16;     // per unit on the busiest worker (query load, pipeline fill and drain,
                        // output store: about six pages of steps), pages * 16
  int32_t split_x16;    // per split unit on the busiest worker (partial write), pages * 16
  int32_t combine_x16;  // per partial, spread over the workers (combine read), pages * 16
};

constexpr PlanCosts kPlanCosts = {96, 32, 48};
constexpr int kNumCandidates = 96;

SPLASH_HD int32_t tile_keys(int32_t seq_len, int32_t q_chunk, int32_t i) {
  return seq_len - q_chunk + i + 1;
}

SPLASH_HD int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

// Division of 32-bit unsigned n by an invariant divisor 1 <= d <= 2^31 with
// one multiply-high (Granlund and Montgomery, 1994; the round-up magic with
// the extra add step): for 2^(l-1) < d <= 2^l, m = floor(2^32 (2^l - d) / d)
// + 1 and t = mulhi(m, n) give floor(n / d) = (t + ((n - t) >> 1)) >> (l - 1)
// for every 32-bit n.  d = 1 is passed through.
struct UDiv {
  uint32_t m, s, d;
};
SPLASH_HD UDiv udiv_make(uint32_t d) {
  UDiv r;
  r.d = d;
  r.m = 0;
  r.s = 0;
  if (d >= 2) {
    const uint32_t l = 32u - (uint32_t)__builtin_clz(d - 1u);  // ceil(log2 d)
    r.m = (uint32_t)(((uint64_t)((1ull << l) - d) << 32) / d + 1u);
    r.s = l - 1u;
  }
  return r;
}
SPLASH_HD uint32_t udiv(uint32_t n, UDiv v) {
  const uint32_t t = (uint32_t)(((uint64_t)v.m * n) >> 32);
  const uint32_t q = (t + ((n - t) >> 1)) >> v.s;
  return v.d == 1u ? n : q;  // a select, no branch
}

// ceil(a / b) for a >= 0, b >= 1, with a 32-bit division whenever it fits.
SPLASH_HD int64_t ceil_div_u(int64_t a, int32_t b) {
  if (a < 0x7fffffffLL - b) return (int64_t)(((uint32_t)a + (uint32_t)b - 1u) / (uint32_t)b);
  return (a + b - 1) / b;
}

// Candidate unit size k (0-based): ceil(maxP / parts_k) with parts_k = k + 1
// for k < 64, then a geometric continuation (parts_{k} = parts_{k-1} +
// parts_{k-1} / 8 from parts_63 = 64) so very long tiles can be cut finely.
SPLASH_HD int32_t plan_candidate_parts(int32_t k) {
  int32_t parts = k + 1;
  if (k >= 64) {
    parts = 64;
    for (int32_t j = 64; j <= k; ++j) parts += parts / 8;
  }
  return parts;
}
// (cap: the largest unit, kMaxUnitPages, or smaller for the top-k variant,
// whose unit holds its selected rows' addresses in the same LDS)
SPLASH_HD int32_t plan_candidate_size(int32_t parts, int32_t max_pages, int32_t cap = kMaxUnitPages) {
  int32_t c = ceil_div(max_pages, parts);
  if (c > cap) c = cap;
  return c < 1 ? 1 : c;
}
SPLASH_HD int32_t plan_candidate(int32_t k, int32_t max_pages) {
  return plan_candidate_size(plan_candidate_parts(k), max_pages);
}

// Estimated step time of unit size c (page equivalents * 16 * G), given the
// number of units W and split units S it produces.
SPLASH_HD int64_t plan_cost(int32_t c, int64_t W, int64_t S, int64_t total_pages,
                            int32_t max_pages, int32_t G, PlanCosts k) {
  const int64_t R = ceil_div_u(W, G);                      // units on the busiest worker
  const int64_t RS = ceil_div_u(S, G);                     // split units on it, at most R
  const int64_t c_eff = c < max_pages ? c : max_pages;
  const int64_t mean = total_pages * 16;
  // Busiest worker: at most R units of at most c_eff pages, never below the
  // mean.  (The queue deals the longest units first; a finer estimate of
  // that packing favoured splitting batches of short histories, but measured
  // the saving did not cover the partial writes and the combine.)
  int64_t busy = R * c_eff * 16 * G;
  if (busy < mean) busy = mean;
  return busy + R * k.unit_x16 * G + (RS < R ? RS : R) * k.split_x16 * G + S * k.combine_x16;
}

// Unit u (0-based) of a tile of P pages cut into n units: [P*u/n, P*(u+1)/n).
SPLASH_HD int32_t unit_begin(int32_t P, int32_t n, int32_t u) {
  if (P < 46341) return (int32_t)(((uint32_t)P * (uint32_t)u) / (uint32_t)n);  // product fits in 31 bits
  return (int32_t)(((int64_t)P * u) / n);
}

// ----------------------------------------------------------- fold plan --
//
// For at most one tile per worker (T <= G) the second kind of plan keeps
// tiles whole except the longest.  Ranks r = 0 .. G-1 order the tiles by
// pages, longest first (the host mirror breaks ties by tile index, the
// device in whatever order its atomics give: a tie decides only which worker
// runs which of two equal units), with q_r = 0 for the ranks
// T .. G-1 that have no tile; worker r runs rank r's tile.  For a cap C every
// tile with q_j > C ("long", ranks j < nl) keeps its first C pages and hands
// the rest, its tail, to worker G-1-j: an idle worker, or the one with the
// j-th shortest tile.  That needs 2 nl <= G.  In pages * 16, with U the fixed
// cost of a unit, the busiest worker then runs
//     max(16 C + U,  max_{j < nl} 16 (q_{G-1-j} + q_j - C) + U + U [q_{G-1-j} > 0])
// and every long tile leaves two partials for the combine.  C is chosen over
// 1 .. q_0 - 1 by the same estimate as the unit size (ties to the larger C),
// and the fold plan is taken when it beats every unit size.  Every piece is
// at most max_pages, so the fold needs max_pages <= kMaxUnitPages.

// Estimated step time of cap C given pages by rank q[0..G), or INT64_MAX if
// infeasible (a partner would be long, or the partials exceed max_partials);
// *nl_out = long tiles.
template <typename Q>
SPLASH_HD int64_t fold_cost(int32_t C, const Q& q, int32_t G, int32_t max_partials, PlanCosts k,
                            int32_t* nl_out) {
  int64_t mk = 16 * (int64_t)C + k.unit_x16;
  int32_t nl = 0;
  while (nl < G && q[nl] > C) {
    const int32_t j = nl++;
    if (2 * nl > G || 2 * nl > max_partials) return INT64_MAX;
    const int32_t qk = q[G - 1 - j];
    const int64_t pair = 16 * (int64_t)(qk + q[j] - C) + k.unit_x16 + (qk > 0 ? k.unit_x16 : 0);
    mk = pair > mk ? pair : mk;
  }
  *nl_out = nl;
  return (int64_t)G * (mk + k.split_x16) + 2 * (int64_t)nl * k.combine_x16;
}

// The fold plan is considered for T <= G <= max_workers tiles of at most
// kMaxUnitPages pages, at least one of them longer than a page, and only
// when it could beat the best unit size: every cap cuts the longest tile in
// two, so the busiest worker runs at least half of it (and at least the
// mean), a lower bound on every fold's estimate.
SPLASH_HD bool fold_applicable(int32_t T, int32_t G, int32_t max_workers, int32_t max_pages, int64_t total_pages,
                               int64_t best_cost, PlanCosts k, int32_t cap = kMaxUnitPages) {
  if (!(T >= 1 && T <= G && G <= max_workers && max_pages >= 2 && max_pages <= cap)) return false;
  int64_t busy = 8 * (int64_t)max_pages + k.unit_x16;
  const int64_t mean = 16 * total_pages / G;
  if (mean > busy) busy = mean;
  return (int64_t)G * (busy + k.split_x16) < best_cost;
}

}  // namespace splash
