// plan.h -- host-side layouts and work plans of a reified KB (internal).
//
// A reified KB (Sec. 2.3) is three sparse matrices with one nonzero per row:
// M_subj, M_obj and M_rel map triple l to its subject, object and relation.
// Each of the library's three passes is a segmented sum over the triples
// grouped by one of those ids:
//   forward  Y  : rows = objects,   gathers X[s] and R[r]   (Eq. 4)
//   backward dX : rows = subjects,  gathers dY[o] and R[r]
//   backward dR : rows = relations, gathers X[s] and dY[o]
// so the planner sorts the triples three ways (counting sorts, stable) and
// cuts every row into pieces of at most `piece_len` triples.  A row that fits
// in one piece is written directly by the lane group that sums it; a longer
// row writes one double-precision partial per piece into a workspace slot and
// the partials are added up in piece order by combine tasks, at most
// `fan_in` slots per task, over as many levels as the row needs.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace kbf {

enum LayoutKind { BY_OBJ = 0, BY_SUBJ = 1, BY_REL = 2 };

// One unit of work for a lane group: triples [start, start + len) of the
// layout; dst >= 0 is the output row, dst < 0 is workspace slot -(dst + 1).
struct Piece {
  int32_t start, len, dst, pad;
};

// Sum slots [first, first + n) in order into dst (row if >= 0, else slot -(dst + 1)).
struct CombineTask {
  int32_t first, n, dst, pad;
};

struct LayoutHost {
  int64_t rows = 0;
  std::vector<int32_t> offsets;   // rows + 1
  std::vector<int32_t> col_a;     // gathered id of the first operand, per position
  std::vector<int32_t> col_b;     // id of the second operand, per position
  std::vector<float> weight;      // per position, empty for a hard KB
  std::vector<int32_t> perm;      // caller index of the triple at each position
};

struct PlanHost {
  int32_t piece_len = 0;
  int32_t fan_in = 0;
  std::vector<Piece> pieces;      // longest first
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

// Cuts a layout's rows into pieces and plans the combine levels.
PlanHost plan_layout(const LayoutHost &layout, int32_t piece_len, int32_t fan_in);

}  // namespace kbf
