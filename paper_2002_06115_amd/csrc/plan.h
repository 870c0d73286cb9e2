// plan.h -- host-side layouts and work plans of a reified KB (internal).
//
// A reified KB (Sec. 2.3) is three sparse matrices with one nonzero per row:
// M_subj, M_obj and M_rel map triple l to its subject, object and relation.
// Each of the library's three passes is a segmented sum over the triples
// grouped by one of those ids:
//   forward  Y  : rows = objects,   sum over r-runs of R[r] (.) sum X[s]   (Eq. 4)
//   backward dX : rows = subjects,  sum over r-runs of R[r] (.) sum dY[o]
//   backward dR : rows = relations, sum over s-runs of X[s] (.) sum dY[o]
// so the planner sorts the triples three ways (counting sorts, stable) and
// cuts the sorted list into equal chunks, one per lane group, whatever the
// row lengths (Zipf hubs and one-triple rows alike).  A row inside one chunk
// is written directly by the lane group that sums it; a row that crosses chunk
// boundaries writes one double-precision partial per chunk into a workspace
// slot and the partials are added up in chunk order by combine tasks, at most
// `fan_in` slots per task, over as many levels as the row needs.
#pragma once

#include <climits>
#include <cstdint>
#include <string>
#include <vector>

namespace kbf {

enum LayoutKind { BY_OBJ = 0, BY_SUBJ = 1, BY_REL = 2 };

// Marks a position whose running sum is not written out.
constexpr int32_t kNoFlush = INT32_MIN;

// Sum slots [first, first + n) in order into dst (row if >= 0, else slot -(dst + 1)).
struct CombineTask {
  int32_t first, n, dst, pad;
};

struct LayoutHost {
  int64_t rows = 0;
  std::vector<int32_t> offsets;   // rows + 1
  std::vector<int32_t> col_a;     // id of the operand gathered for every triple (A)
  std::vector<int32_t> col_b;     // id of the operand read once per run (B)
  std::vector<float> weight;      // per position, empty for a hard KB
  std::vector<int32_t> perm;      // caller index of the triple at each position
};

// The stream plan of one layout: the sorted positions are cut into chunks of
// `chunk` consecutive positions, one chunk per lane group.  flush[p] says what
// the lane group does after adding position p: nothing (kNoFlush), write the
// row it just finished (>= 0), or write its partial sum of a row that crosses
// a chunk boundary to workspace slot -(flush[p] + 1).  A row's partials are
// numbered in chunk order and summed in that order by the combine levels.
// Inside a row the positions form runs of equal col_b; run_end[p] marks the
// last position of a run (a row end or chunk end also ends a run), where the
// kernel multiplies the run's sum of A rows by the B row once.
struct PlanHost {
  int32_t chunk = 0;
  int32_t fan_in = 0;
  int64_t n_chunks = 0;
  std::vector<int32_t> flush;      // per position
  std::vector<uint8_t> run_end;    // per position: last of a run of equal col_b (or of a chunk)
  std::vector<int32_t> empty_rows;
  std::vector<std::vector<CombineTask>> levels;
  int64_t n_slots = 0;
  int64_t n_split_rows = 0;
  int64_t max_row_len = 0;
};

// Returns "" when the triple arrays are valid, else a message; *range_error
// tells an out-of-range id (KB_ERANGE) from any other problem (KB_EINVAL).
std::string validate_triples(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                             const int32_t *subj, const int32_t *rel, const int32_t *obj,
                             bool *range_error);

// Builds the three layouts.  keep_perm keeps the caller-index permutation.
void build_layouts(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                   const int32_t *subj, const int32_t *rel, const int32_t *obj,
                   const float *weight, bool keep_perm, LayoutHost out[3]);

// Cuts a layout into chunks, marks the flush points and plans the combine levels.
PlanHost plan_layout(const LayoutHost &layout, int32_t chunk, int32_t fan_in);

}  // namespace kbf
