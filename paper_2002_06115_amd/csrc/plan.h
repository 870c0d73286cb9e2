// plan.h -- host-side layouts and work plans of a reified KB (internal).
//
// A reified KB (Sec. 2.3) is three sparse matrices with one nonzero per row:
// M_subj, M_obj and M_rel map triple l to its subject, object and relation.
// Each of the library's three passes is a segmented sum over the triples
// grouped by one of those ids:
//   forward  Y  : rows = objects,   sum over r-runs of R[r] (.) sum X[s]   (Eq. 4)
//   backward dX : rows = subjects,  sum over r-runs of R[r] (.) sum dY[o]
//   backward dR : rows = relations, sum over s-runs of X[s] (.) sum dY[o]
// so the planner sorts the triples three ways (stable sorts) and
// turns each sorted list into a stream of 8-byte entries cut into equal
// chunks (see PlanHost).
#pragma once

#include <climits>
#include <cstdint>
#include <string>
#include <vector>

namespace kbf {

enum LayoutKind { BY_OBJ = 0, BY_SUBJ = 1, BY_REL = 2 };

// Sum slots [first, first + n) in order into dst (row if >= 0, else slot -(dst + 1)).
struct CombineTask {
  int32_t first, n, dst, pad;
};

struct LayoutHost {
  int64_t rows = 0;
  std::vector<int32_t> row;       // row id of every position (non-decreasing)
  std::vector<int32_t> offsets;   // rows + 1 boundaries, only when asked for (O(rows))
  std::vector<int32_t> col_a;     // id of the operand gathered for every triple (A)
  std::vector<int32_t> col_b;     // id of the operand read once per run (B)
  std::vector<float> weight;      // per position, empty for a hard KB
  std::vector<int32_t> perm;      // caller index of the triple at each position
};

// One 8-byte stream entry.  A triple: x = (id gathered for this triple, col_a)
// | kRunStart when it is the first triple of a run of equal col_b since the
// last marker, y = col_b | kSameA when the entry right before it is a triple
// of the same row with the same col_a and both lie in one kernel step of
// kStepEntries entries (the kernel then reuses that entry's gathered row
// instead of reading it again).  A marker (x = kMarker): write the running
// sum to y -- a row (y >= 0), a workspace slot -(y + 1), or nothing
// (y = kNoTarget) -- and restart from zero.
struct Entry {
  int32_t x, y;
};
constexpr int32_t kMarker = -1;
constexpr int32_t kRunStart = 1 << 30;
constexpr int32_t kSameA = 1 << 30;
constexpr int32_t kIdMask = kRunStart - 1;
constexpr int32_t kNoTarget = INT32_MIN;
// Entries a lane group takes per kernel step (the stream kernel's unroll):
// chunks start at multiples of it, so steps are aligned in the stream.
constexpr int32_t kStepEntries = 8;

// The stream plan of one layout.  The sorted triples of every non-empty row
// are followed by a marker that writes the row, and the stream is cut into
// chunks of `chunk` entries, one chunk per lane group, whatever the row
// lengths (Zipf hubs and one-triple rows alike); the stream is padded with
// no-op markers to whole chunks.  The last entry of every chunk is a marker:
// where a row continues past it, that marker writes the chunk's partial sum of
// the row to a workspace slot, and the row's final marker writes its last
// partial to a slot too.  A row's slots are numbered
// consecutively in chunk order and summed in that order by combine tasks, at
// most `fan_in` slots per task, over as many levels as the row needs.
// Inside a row the triples form runs of equal col_b; the kernel reads a run's
// B row once, at the entry flagged kRunStart, and keeps it for the run.
// Rows no triple reaches, as pieces of consecutive rows [first, first + count),
// count <= kEmptyPiece: one zero-fill task each.
struct EmptyPiece {
  int32_t first, count;
};
constexpr int32_t kEmptyPiece = 4096;

// Chunk lists: the stream is cut into n_xcd consecutive lists of whole
// chunks, list x for the workgroups that run on XCD x (workgroup w runs on
// XCD w mod 8 on an MI355X), so that each XCD's L2 caches the rows its own
// triples gather.  The gathered ids (or, with class_by_b, the second
// operand's) are split into n_xcd classes of about equal weight; a row with
// at least hub_min triples is cut into one segment per class present, each
// in its class's list (its partial sums go to slots and are combined like
// those of a row that crosses chunks), and every other row goes whole into
// one list (the class of its first triple, unless that list is already
// full).  Inside a hub segment the triples are ordered
// by gathered id (hub_by_a) or by (second operand, gathered id), and a
// list's hub chunks are ordered by their first gathered id (band), so that
// the chunks in flight at once gather from nearby rows.  The order of
// chunks never changes a result: each chunk's sums and targets are fixed.
constexpr int kMaxXcd = 8;
struct PlanOptions {
  int32_t chunk = 256;
  int32_t fan_in = 32;
  int32_t n_xcd = 1;       // chunk lists (1: a single list in row order)
  int64_t hub_min = 256;   // rows with at least this many triples are split by class
  bool hub_by_a = true;
  bool band = true;
  int64_t n_ids_a = 0;     // size of the gathered id space
  // Classes of the second operand's ids instead of the gathered ones (every
  // run of equal second operand then stays in one list).
  bool class_by_b = false;
  int64_t n_ids_b = 0;     // size of the second operand's id space
  // With hub_by_a false: hub segments ordered by (block of the gathered id,
  // second operand, gathered id), the gathered ids cut into a_blocks equal
  // ranges (0 or 1: no blocks), so that with band the chunks of a list walk
  // the gathered table one block at a time.
  int32_t a_blocks = 0;
};

struct PlanHost {
  int32_t chunk = 0;
  int32_t fan_in = 0;
  int64_t n_chunks = 0;
  int32_t n_xcd = 1;
  std::vector<int64_t> xcd_chunk;   // n_xcd + 1 boundaries of the chunk lists
  std::vector<Entry> entries;
  std::vector<float> weights;       // per entry (markers 0), empty for a hard KB
  std::vector<EmptyPiece> empty;    // the rows no triple reaches
  int64_t n_empty_rows = 0;
  std::vector<std::vector<CombineTask>> levels;
  int64_t n_slots = 0;
  int64_t n_split_rows = 0;
  int64_t max_row_len = 0;
};

// The share of the entries of `col` (ids below n_ids) whose id is one of the
// ceil(frac * n_ids) most frequent ones: how skewed the id distribution is.
double top_id_share(const std::vector<int32_t> &col, int64_t n_ids, double frac);

// Returns "" when the triple arrays are valid, else a message; *range_error
// tells an out-of-range id (KB_ERANGE) from any other problem (KB_EINVAL).
std::string validate_triples(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                             const int32_t *subj, const int32_t *rel, const int32_t *obj,
                             bool *range_error);

// How build_layouts sorts: kAuto takes the radix sort of a 64-bit key per
// triple when 2 * bits(N_E - 1) + bits(N_R - 1) <= 64, else chained counting
// sorts; kCounting forces the latter (both give the same stable orders).
enum class LayoutSort { kAuto, kCounting };

// Builds the three layouts.  keep_perm keeps the caller-index permutation,
// keep_offsets the per-row boundaries (O(rows); the plans do not need them).
// Everything else is O(N_T) plus, for dense id spaces, O(N_E + N_R).
void build_layouts(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                   const int32_t *subj, const int32_t *rel, const int32_t *obj,
                   const float *weight, bool keep_perm, bool keep_offsets, LayoutHost out[3],
                   LayoutSort how = LayoutSort::kAuto);

// Cuts a layout into chunk lists, marks the flush points and plans the
// combine levels.
PlanHost plan_layout(const LayoutHost &layout, const PlanOptions &options);
// One list in row order (n_xcd = 1).
PlanHost plan_layout(const LayoutHost &layout, int32_t chunk, int32_t fan_in);

}  // namespace kbf
