// Host planner under AddressSanitizer and UndefinedBehaviorSanitizer: the
// validation, the three stable sorts and the stream plans of
// random, Zipf-hub, empty and degenerate KBs, with the plan's invariants
// checked along the way.  Exit status 0 when every check holds (sanitizer
// reports abort the program).  Built and run by tests/test_host_sanitizers.py.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "plan.h"

using namespace kbf;

static int failures = 0;
#define CHECK(cond, ...)                                  \
  do {                                                    \
    if (!(cond)) {                                        \
      std::fprintf(stderr, "check failed: %s: ", #cond);  \
      std::fprintf(stderr, __VA_ARGS__);                  \
      std::fprintf(stderr, "\n");                         \
      ++failures;                                         \
    }                                                     \
  } while (0)

// Every stream property the kernels rely on.
static void check_plan(const LayoutHost &L, const PlanHost &P, int32_t chunk, const char *what) {
  const int64_t n = (int64_t)P.entries.size();
  CHECK(n % chunk == 0, "%s: %lld entries, chunk %d", what, (long long)n, chunk);
  CHECK(P.n_chunks * chunk == n, "%s: n_chunks", what);
  int64_t triples = 0, row_markers = 0;
  std::vector<int> slot_written(P.n_slots, 0);
  for (int64_t p = 0; p < n; ++p) {
    const Entry &e = P.entries[p];
    if (p % chunk == chunk - 1) CHECK(e.x == kMarker, "%s: chunk end %lld is no marker", what, (long long)p);
    if (e.x == kMarker) {
      if (e.y >= 0) {
        CHECK(e.y < L.rows, "%s: row target %d", what, e.y);
        ++row_markers;
      } else if (e.y != kNoTarget) {
        const int64_t slot = -(int64_t)e.y - 1;
        CHECK(slot >= 0 && slot < P.n_slots, "%s: slot %lld", what, (long long)slot);
        if (slot >= 0 && slot < P.n_slots) ++slot_written[slot];
      }
    } else {
      CHECK(e.x >= 0, "%s: entry %lld", what, (long long)p);
      ++triples;
    }
  }
  CHECK(triples == (int64_t)L.col_a.size(), "%s: %lld of %zu triples in the stream", what,
        (long long)triples, L.col_a.size());
  int64_t non_empty = 0;
  for (size_t p = 0; p < L.row.size(); ++p) non_empty += p == 0 || L.row[p] != L.row[p - 1];
  CHECK(row_markers + P.n_split_rows == non_empty, "%s: row markers", what);
  CHECK(P.n_empty_rows == L.rows - non_empty, "%s: empty rows", what);
  // The empty pieces cover exactly the rows without triples, in order.
  std::vector<char> has(L.rows, 0);
  for (int32_t q : L.row) has[q] = 1;
  int64_t covered = 0, last_end = 0;
  for (const EmptyPiece &e : P.empty) {
    CHECK(e.count >= 1 && e.count <= kEmptyPiece && e.first >= last_end &&
              (int64_t)e.first + e.count <= L.rows,
          "%s: empty piece (%d, %d)", what, e.first, e.count);
    for (int32_t q = e.first; q < e.first + e.count && q < L.rows; ++q)
      CHECK(!has[q], "%s: row %d has triples but is in an empty piece", what, q);
    covered += e.count;
    last_end = (int64_t)e.first + e.count;
  }
  CHECK(covered == P.n_empty_rows, "%s: empty pieces cover %lld rows", what, (long long)covered);
  // Every stream slot is written once; combine outputs are later slots.
  int64_t stream_slots = 0;
  for (int64_t s = 0; s < P.n_slots; ++s) {
    CHECK(slot_written[s] <= 1, "%s: slot %lld written twice", what, (long long)s);
    stream_slots += slot_written[s];
  }
  int64_t tasks_to_rows = 0;
  for (const auto &level : P.levels)
    for (const CombineTask &t : level) {
      CHECK(t.n >= 1 && t.n <= P.fan_in, "%s: task of %d slots", what, t.n);
      CHECK(t.first >= 0 && t.first + t.n <= P.n_slots, "%s: task range", what);
      if (t.dst >= 0) {
        CHECK(t.dst < L.rows, "%s: task row", what);
        ++tasks_to_rows;
      } else {
        CHECK(-(int64_t)t.dst - 1 < P.n_slots, "%s: task slot", what);
      }
    }
  CHECK(tasks_to_rows == P.n_split_rows, "%s: final combine tasks", what);
  if (!P.weights.empty()) CHECK(P.weights.size() == P.entries.size(), "%s: weights", what);
}

// Runs the plan on the CPU with an exact integer value per triple, chunk by
// chunk as the stream kernel does (a run's second operand is taken from its
// first triple), then the combine levels in order, and compares every row's
// total with a direct sum over the layout: each triple counted once, into its
// own row, whatever the lists and the chunk order.
static void interpret_plan(const LayoutHost &L, const PlanHost &P, int32_t chunk,
                           const char *what) {
  auto val = [](int32_t a, int32_t b) -> int64_t {
    return (int64_t)(a % 1009) * 1013 + (int64_t)(b % 997) + 1;
  };
  std::vector<int64_t> want(L.rows, 0), got(L.rows, 0), slot(P.n_slots, 0);
  std::vector<int> writes(L.rows, 0);
  for (size_t p = 0; p < L.col_a.size(); ++p) want[L.row[p]] += val(L.col_a[p], L.col_b[p]);
  CHECK((int64_t)P.xcd_chunk.size() == P.n_xcd + 1 && P.xcd_chunk.front() == 0 &&
            P.xcd_chunk.back() == P.n_chunks,
        "%s: chunk lists", what);
  for (size_t x = 1; x < P.xcd_chunk.size(); ++x)
    CHECK(P.xcd_chunk[x - 1] <= P.xcd_chunk[x], "%s: chunk list %zu", what, x);
  for (int64_t c = 0; c < P.n_chunks; ++c) {
    int64_t acc = 0;
    bool held = false;
    int32_t hb = 0;
    int32_t held_a = -1;  // the A row the previous entry gathered (or reused)
    for (int64_t p = c * chunk; p < (c + 1) * chunk; ++p) {
      const Entry &e = P.entries[p];
      if (e.x >= 0) {
        const int32_t b = e.y & kIdMask;
        int32_t a = e.x & kIdMask;
        if (e.y & kSameA) {
          // The kernel skips this gather and takes the previous entry's row:
          // only inside a step, after a triple with the same id.
          CHECK(p % kStepEntries != 0 && held_a == a,
                "%s: entry %lld reuses a row it may not (step start or other id)", what,
                (long long)p);
          a = held_a;
        }
        if (e.x & kRunStart) {
          hb = b;
          held = true;
        }
        CHECK(held && hb == b, "%s: entry %lld outside a run of its second operand", what,
              (long long)p);
        acc += val(a, b);
        held_a = a;
      } else {
        held_a = -1;
        if (e.y >= 0 && e.y < L.rows) {
          got[e.y] += acc;
          ++writes[e.y];
        } else if (e.y != kNoTarget && -(int64_t)e.y - 1 < P.n_slots) {
          slot[-(int64_t)e.y - 1] = acc;
        }
        acc = 0;
        held = false;
      }
    }
  }
  for (const auto &level : P.levels)
    for (const CombineTask &t : level) {
      int64_t sum = 0;
      for (int32_t i = 0; i < t.n; ++i)
        if (t.first + i < P.n_slots) sum += slot[t.first + i];
      if (t.dst >= 0 && t.dst < L.rows) {
        got[t.dst] += sum;
        ++writes[t.dst];
      } else if (t.dst < 0 && -(int64_t)t.dst - 1 < P.n_slots) {
        slot[-(int64_t)t.dst - 1] = sum;
      }
    }
  std::vector<char> has(L.rows, 0);
  for (int32_t q : L.row) has[q] = 1;
  for (int64_t q = 0; q < L.rows; ++q) {
    CHECK(got[q] == want[q], "%s: row %lld sums to %lld, want %lld", what, (long long)q,
          (long long)got[q], (long long)want[q]);
    CHECK(writes[q] == (has[q] ? 1 : 0), "%s: row %lld written %d times", what, (long long)q,
          writes[q]);
  }
}

static void check_layout(const LayoutHost &L, int64_t n_t, const char *what) {
  CHECK((int64_t)L.col_a.size() == n_t && (int64_t)L.col_b.size() == n_t &&
            (int64_t)L.row.size() == n_t,
        "%s: sizes", what);
  CHECK((int64_t)L.offsets.size() == L.rows + 1 && L.offsets[0] == 0 && L.offsets[L.rows] == n_t,
        "%s: offsets", what);
  for (int64_t q = 0; q < L.rows; ++q) {
    CHECK(L.offsets[q] <= L.offsets[q + 1], "%s: offsets not monotone", what);
    for (int32_t p = L.offsets[q]; p < L.offsets[q + 1]; ++p) {
      CHECK(L.row[p] == q, "%s: row id of position %d", what, p);
      if (p > L.offsets[q])
        CHECK(L.col_b[p - 1] <= L.col_b[p], "%s: runs not sorted in row %lld", what, (long long)q);
    }
  }
}

static void run_case(const char *what, int64_t n_e, int64_t n_r, std::vector<int32_t> s,
                     std::vector<int32_t> r, std::vector<int32_t> o, bool weighted) {
  const int64_t n_t = (int64_t)s.size();
  bool range = false;
  CHECK(validate_triples(n_e, n_r, n_t, s.data(), r.data(), o.data(), &range).empty(),
        "%s: valid triples refused", what);
  std::vector<float> w;
  if (weighted) {
    w.resize(n_t);
    for (int64_t l = 0; l < n_t; ++l) w[l] = 0.5f + (float)(l % 7);
  }
  LayoutHost L[3], C[3];
  build_layouts(n_e, n_r, n_t, s.data(), r.data(), o.data(), weighted ? w.data() : nullptr, true,
                true, L);
  // The chained counting sorts give the same stable orders.
  build_layouts(n_e, n_r, n_t, s.data(), r.data(), o.data(), weighted ? w.data() : nullptr, true,
                true, C, LayoutSort::kCounting);
  for (int k = 0; k < 3; ++k) {
    CHECK(L[k].rows == C[k].rows && L[k].row == C[k].row && L[k].col_a == C[k].col_a &&
              L[k].col_b == C[k].col_b && L[k].weight == C[k].weight && L[k].perm == C[k].perm &&
              L[k].offsets == C[k].offsets,
          "%s: layout %d differs between the radix and the counting sorts", what, k);
    check_layout(L[k], n_t, what);
    for (int32_t chunk : {16, 24, 256}) {
      for (int32_t fan_in : {2, 3, 32}) {
        const PlanHost P = plan_layout(L[k], chunk, fan_in);
        check_plan(L[k], P, chunk, what);
        interpret_plan(L[k], P, chunk, what);
      }
      // One chunk list per XCD, hub rows split by class of the gathered id
      // (or of the second operand), and hub segments led by blocks of the
      // gathered id.
      for (int64_t hub_min : {int64_t(4), int64_t(64)})
        for (bool by_a : {true, false})
          for (bool band : {true, false})
            for (bool class_b : {false, true})
              for (int32_t blocks : {0, 5}) {
                if (by_a && blocks) continue;  // blocks order only (second operand, id) segments
                PlanOptions po;
                po.a_blocks = blocks;
                po.chunk = chunk;
                po.fan_in = 3;
                po.n_xcd = 8;
                po.hub_min = hub_min;
                po.hub_by_a = by_a;
                po.band = band;
                po.n_ids_a = n_e;
                po.class_by_b = class_b;
                po.n_ids_b = k == 2 ? n_e : n_r;  // dR's second operand is the subject
                const PlanHost P = plan_layout(L[k], po);
                check_plan(L[k], P, chunk, what);
                interpret_plan(L[k], P, chunk, what);
              }
    }
  }
}

int main() {
  std::mt19937_64 g(20020615);
  // Invalid arguments: each refused with a message, range errors flagged.
  {
    std::vector<int32_t> s = {0, 5}, r = {0, 0}, o = {1, 1};
    bool range = false;
    CHECK(!validate_triples(5, 1, 2, s.data(), r.data(), o.data(), &range).empty() && range,
          "subject id == N_E accepted");
    CHECK(!validate_triples(-1, 1, 0, nullptr, nullptr, nullptr, &range).empty() && !range,
          "negative N_E accepted");
    CHECK(!validate_triples(5, 1, 2, nullptr, r.data(), o.data(), &range).empty(),
          "null subj accepted");
    CHECK(!validate_triples((1 << 30) + 1, 1, 0, nullptr, nullptr, nullptr, &range).empty(),
          "N_E above 2^30 accepted");
  }
  // The skew statistic that picks dR's classing.
  {
    const std::vector<int32_t> col = {0, 0, 0, 1, 2, 3, 3, 0};
    CHECK(top_id_share(col, 4, 0.25) == 0.5, "top 1 of 4 ids: half the entries");
    CHECK(top_id_share(col, 4, 0.5) == 6.0 / 8.0, "top 2 of 4 ids: six of eight entries");
    CHECK(top_id_share(col, 4, 1.0) == 1.0, "every id: every entry");
    CHECK(top_id_share(col, 100, 0.01) == 0.5, "top 1 of 100 ids (one rounded up)");
    CHECK(top_id_share({}, 4, 0.5) == 0.0, "no entries");
  }
  // Random KBs.
  for (int rep = 0; rep < 4; ++rep) {
    const int64_t n_e = 50 + rep * 300, n_r = 1 + rep * 3, n_t = 2000 + rep * 5000;
    std::uniform_int_distribution<int32_t> E(0, (int32_t)n_e - 1), R(0, (int32_t)n_r - 1);
    std::vector<int32_t> s(n_t), r(n_t), o(n_t);
    for (int64_t l = 0; l < n_t; ++l) {
      s[l] = E(g);
      r[l] = R(g);
      o[l] = E(g);
    }
    run_case("random", n_e, n_r, s, r, o, rep % 2 == 1);
  }
  // One hub holding every triple, beside empty rows; duplicate triples.
  {
    const int64_t n_t = 20000;
    std::vector<int32_t> s(n_t, 3), r(n_t), o(n_t);
    for (int64_t l = 0; l < n_t; ++l) {
      r[l] = (int32_t)(l % 2);
      o[l] = (int32_t)(l % 5);
    }
    run_case("hub", 10, 2, s, r, o, true);
  }
  // Rows of 2^16 triples or more: their class segments are ordered by the
  // radix sort (shorter hub rows by a sort of key / position pairs).
  {
    const int64_t n_t = 70000;
    std::uniform_int_distribution<int32_t> E(0, 4999);
    std::vector<int32_t> s(n_t, 3), r(n_t, 0), o(n_t);
    for (int64_t l = 0; l < n_t; ++l) o[l] = l % 2 ? E(g) : (int32_t)(l % 11);
    run_case("long hub", 5000, 1, s, r, o, false);
  }
  // Sparse id space: few triples over many ids (the comparison-sort path).
  {
    const int64_t n_e = 1 << 20, n_t = 3000;
    std::uniform_int_distribution<int32_t> E(0, (int32_t)n_e - 1);
    std::vector<int32_t> s(n_t), r(n_t), o(n_t);
    for (int64_t l = 0; l < n_t; ++l) {
      s[l] = l % 3 ? E(g) : (int32_t)(n_e - 1 - l % 5);
      r[l] = (int32_t)(l % 4);
      o[l] = l % 2 ? E(g) : (int32_t)(l % 7);
    }
    run_case("sparse ids", n_e, 4, s, r, o, true);
  }
  // Keys of exactly 64 bits (2 * 21 + 22 bits): the widest KB the radix sort
  // takes, with the largest ids in every field; one relation more and the
  // counting sorts take over.
  for (int64_t n_r : {int64_t(1) << 22, (int64_t(1) << 22) + 1}) {
    const int64_t n_e = int64_t(1) << 21, n_t = 5000;
    std::uniform_int_distribution<int32_t> E(0, (int32_t)n_e - 1), R(0, (int32_t)n_r - 1);
    std::vector<int32_t> s(n_t), r(n_t), o(n_t);
    for (int64_t l = 0; l < n_t; ++l) {
      s[l] = l % 4 ? E(g) : (int32_t)(n_e - 1);
      r[l] = l % 5 ? R(g) : (int32_t)(n_r - 1);
      o[l] = l % 6 ? E(g) : (int32_t)(n_e - 1 - l % 2);
    }
    run_case(n_r == (int64_t(1) << 22) ? "64-bit keys" : "65-bit keys", n_e, n_r, s, r, o, true);
  }
  // Empty KB; one entity with self-loops; one relation.
  run_case("empty", 7, 3, {}, {}, {}, false);
  run_case("self loops", 1, 1, std::vector<int32_t>(100, 0), std::vector<int32_t>(100, 0),
           std::vector<int32_t>(100, 0), false);
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("planner checks passed\n");
  return 0;
}
