// Product schedules of the level GEMMs (host code, no HIP types).
//
// The S digits of an element are the coefficients of a polynomial in
// x = 2^-w (digit 0 most significant), and level t of the product is the
// coefficient of x^t of DA(x) DB(x): G_t = sum over p + q = t of DA_p DB_q
// (section 2, equation (3) and the rewritten product).  A schedule says which
// FP64 GEMMs compute these levels:
//
//  * the pair schedule (the paper's): one GEMM per digit pair (p, q) with
//    p + q <= T, the pairs of a level summed into one output plane;
//  * the Karatsuba schedule: operand "combinations" (sums of digits of one
//    element, e.g. DA_0 + DA_4) are multiplied instead, so that fewer GEMMs
//    cover the same levels (Karatsuba's identity
//    (a0 + a1 x)(b0 + b1 x) = a0 b0 + x [(a0 + a1)(b0 + b1) - a0 b0 - a1 b1] + x^2 a1 b1,
//    applied recursively and truncated at level T).  Each GEMM output plane
//    then enters several levels with small integer coefficients.
//
// Both are exact: digits and their sums are integers, every GEMM partial sum is
// an integer kept below 2^53 by the job budget, and the levels are formed from
// the planes in 64-bit integers.  So both schedules give bit-identical levels.
#pragma once

#include <cstdint>
#include <vector>

namespace mdg {

// Digits a Karatsuba combination may draw on (digit sets are 64-bit masks);
// products with more digits per element keep the pair schedule.
constexpr int kMaxComboDigits = 64;

struct Schedule {
  int S = 0, T = 0;
  bool direct_levels = true;  // plane j of the GEMM output is level job_out[j] (pair schedule)
  int terms = 0;              // GEMMs of length k (digit-combination pairs)
  // Operand combinations: combo c < S is digit c; combo c >= S is the sum of
  // combos par1[c] and par2[c] (disjoint digit sets), created in index order.
  std::vector<uint64_t> mask_a, mask_b;
  std::vector<int> par1_a, par2_a, par1_b, par2_b;
  std::vector<int> depth_a, depth_b;  // 0 for digits, 1 + max(parents) otherwise
  // GEMM jobs (heaviest first): job j sums the products of the combination
  // pairs pairs[job_first[j] .. job_first[j] + job_count[j]) into plane job_out[j].
  std::vector<int> job_first, job_count, job_out;
  std::vector<int> pair_a, pair_b;
  // K split: job j runs k chunk job_chunk[j] of ksplit (empty: the whole k).
  // The chunks of a job write separate planes with the same level entries, and
  // the accumulation adds them (partial sums of integers: exact).
  int ksplit = 1;
  std::vector<int> job_chunk;
  // Levels from planes (Karatsuba schedule): level t = sum over the entries
  // (plane, t, coef) of coef * plane; entries sorted by plane, plane_first[j]
  // indexes the first entry of plane j (size planes + 1).
  int planes = 0;
  std::vector<int> plane_first, entry_level, entry_coef;
  int64_t max_job_weight = 0;  // max over jobs of sum |combo a| |combo b| (digits per combination)
};

// The paper's pair schedule: one job per level t <= T (heaviest first), the
// pairs (p, t - p) of the level in increasing p, plane = level.
Schedule pair_schedule(int S, int T);

// Grouped products (section 3: the numbers grouped by exponent class and, with
// sign, by sign; every group pair multiplied): G = (sign ? 2 : 1) Ge groups of S
// digit panels (group g's digits are combinations g S .. g S + S - 1, on a grid
// g % Ge digits below the line's), every group pair (g, h) keeps its pairs
// p + q <= T at level p + q + g % Ge + h % Ge; one job per level
// t <= T + 2 (Ge - 1), heaviest first, plane = level.  The schedule's S is G S
// and its T is T + 2 (Ge - 1).  Every element lies in one group, so a level sums
// at most max_pairs(S, T) products per k index: the pair schedule's bound.
Schedule group_schedule(int S, int T, int Ge, bool sign);

// One job per pair (p, q) with p + q <= T, written to plane p S + q.
Schedule per_pair_schedule(int S, int T);

// Costs of the parts of a schedule other than its GEMMs, each relative to one
// GEMM term (one k-long product of two combinations over all m x n outputs).
struct ScheduleCosts {
  double plane = 0.0;    // an output plane: written by the GEMM, read by the accumulation
  double entry = 0.0;    // a (plane, level, coefficient) entry applied per output element
  double combo_a = 0.0;  // a combination panel of A (m x k): two panels read, one written
  double combo_b = 0.0;  // a combination panel of B (k x n)
};

// Karatsuba schedule for S digits and cutoff T.  budget: the largest digit
// count product |combo a| |combo b| summed over one job (so that
// k budget (2^w - 1)^2 < 2^53).  Picks, level by level of the recursion, the
// split that minimizes terms + the costs of its planes, entries and
// combinations; returns the pair schedule when that is cheaper overall
// (fallback) or when it has no more terms.
Schedule karatsuba_schedule(int S, int T, int64_t budget, const ScheduleCosts& costs, bool fallback);

// The cost of a schedule in GEMM terms, as karatsuba_schedule counts it.
double schedule_cost(const Schedule& s, const ScheduleCosts& costs);

// The schedule with every job split into `sigma` k chunks (sigma > 1 turns a
// pair schedule into one whose planes enter the levels through entries).
Schedule split_k(const Schedule& s, int sigma);

// Device table of a schedule: 32-bit words
//   [3 J job words: first | count << 16, out plane, chunk | ksplit << 16]
//   [P pair words: a | b << 16]
//   [planes + 1 chunk_first words] [2 words per chunk]
//   [2 words per combination of A: digit set, low word first] [same for B]
// The entries of plane j are chunks chunk_first[j] .. chunk_first[j+1]-1 of
// four 16-bit entries each (level | (uint8)coef << 8, entry i in bits 16 (i%2)
// of word i/2); a plane's last chunk is padded with (trash level, coef 0),
// trash level = T + 1 (a slot the accumulation keeps and never reads).
struct ScheduleTable {
  std::vector<uint32_t> words;
  int64_t jobs_off = 0, pairs_off = 0, chunk_first_off = 0, chunks_off = 0, masks_a_off = 0, masks_b_off = 0;
};
ScheduleTable schedule_table(const Schedule& s);

}  // namespace mdg
