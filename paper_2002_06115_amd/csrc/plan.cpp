// plan.cpp -- host-side layouts and work plans of a reified KB.
//
// The reified KB of Sec. 2.3 keeps, per triple, its subject, object and
// relation ids (the one nonzero of row l in M_subj, M_obj and M_rel).  Here
// the triples are sorted three ways with stable sorts: by (o, r, s), by
// (s, r, o) and by (r, s, o) -- a radix sort of one 64-bit key per triple
// where the three ids fit one, else chained counting sorts over dense id
// spaces and comparison sorts where the id space is far larger than the KB
// -- and the plans are built from the sorted rows alone, so building a KB
// costs O(N_T + number of empty-row ranges) beyond the sorts.  The secondary key
// groups each row into runs of equal second operand (the relation for the
// forward and dX passes, the subject for dR), so the kernels read that
// operand once per run instead of once per triple.
#include "plan.h"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstdio>
#include <exception>
#include <functional>
#include <thread>

namespace kbf {

std::string validate_triples(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                             const int32_t *subj, const int32_t *rel, const int32_t *obj,
                             bool *range_error) {
  *range_error = false;
  char msg[160];
  if (n_entities < 0 || n_relations < 0 || n_triples < 0)
    return "n_entities, n_relations and n_triples must be >= 0";
  if (n_entities > (1 << 30) || n_relations > (1 << 30))
    return "n_entities and n_relations must be at most 2^30";
  if (n_triples > INT32_MAX) return "n_triples must be below 2^31";
  if (n_triples > 0 && (!subj || !rel || !obj)) return "subj, rel and obj must be non-NULL";
  for (int64_t l = 0; l < n_triples; ++l) {
    if (subj[l] < 0 || subj[l] >= n_entities || obj[l] < 0 || obj[l] >= n_entities ||
        rel[l] < 0 || rel[l] >= n_relations) {
      *range_error = true;
      std::snprintf(msg, sizeof msg, "triple %lld = (%d, %d, %d) has an id out of range",
                    (long long)l, subj[l], rel[l], obj[l]);
      return msg;
    }
  }
  return "";
}

// Stable sort of the triple ids in `in` by key[id], key in [0, n_keys), and,
// when `offsets` is given, the row boundaries: (*offsets)[k] = the first
// position with key >= k, for k = 0 .. n_keys.  A counting sort (O(n +
// n_keys), `count` is its reusable scratch) where the key space is comparable
// to the number of ids; a stable comparison sort (O(n log n)) where it is far
// larger, so that a KB of a few triples over 2^30 entity ids costs no pass
// over the whole id space except the offsets themselves.
static void sort_by_key(const int32_t *key, int64_t n_keys, const std::vector<int32_t> &in,
                        std::vector<int32_t> &out, std::vector<int32_t> *offsets,
                        std::vector<int32_t> &count) {
  const int64_t n = (int64_t)in.size();
  out.resize(in.size());
  if (n_keys > 8 * n + 1024) {
    out = in;
    std::stable_sort(out.begin(), out.end(),
                     [key](int32_t a, int32_t b) { return key[a] < key[b]; });
    if (offsets) {
      offsets->resize(n_keys + 1);
      int64_t p = 0;
      for (int64_t k = 0; k <= n_keys; ++k) {
        while (p < n && key[out[p]] < k) ++p;
        (*offsets)[k] = (int32_t)p;
      }
    }
    return;
  }
  count.assign(n_keys + 1, 0);  // n < 2^31, so every count and prefix fits int32
  for (int32_t id : in) ++count[key[id] + 1];
  for (int64_t k = 0; k < n_keys; ++k) count[k + 1] += count[k];
  if (offsets) offsets->assign(count.begin(), count.begin() + (n_keys + 1));
  for (int32_t id : in) out[count[key[id]]++] = id;
}

static void fill_layout(LayoutHost &L, int64_t rows, std::vector<int32_t> &&order,
                        std::vector<int32_t> &&offsets, const int32_t *key, const int32_t *a,
                        const int32_t *b, const float *weight, bool keep_perm) {
  L.rows = rows;
  L.offsets = std::move(offsets);
  const size_t n = order.size();
  L.row.resize(n);
  L.col_a.resize(n);
  L.col_b.resize(n);
  for (size_t p = 0; p < n; ++p) {
    L.row[p] = key[order[p]];
    L.col_a[p] = a[order[p]];
    L.col_b[p] = b[order[p]];
  }
  if (weight) {
    L.weight.resize(n);
    for (size_t p = 0; p < n; ++p) L.weight[p] = weight[order[p]];
  }
  if (keep_perm) L.perm = std::move(order);
}

// Stable LSD radix sort of `key` (11-bit digits, as many passes as the
// largest key has digits), carrying the triple ids along when `id` is
// non-null, on `threads` host threads.  Each pass: every thread counts the
// digits of its contiguous block of the input; the bucket of digit d for
// thread t starts after all smaller digits and after digit d of the threads
// before t, so each thread scatters its block in order and the pass is
// stable, whatever the thread count (the result is the same for any).  A pass
// is a sequential read and a scatter into 2048 buckets, unlike a counting
// sort over an id space of millions, whose gathers and scatters miss the
// caches.
static void radix_sort(std::vector<uint64_t> &key, std::vector<int32_t> *id, int threads) {
  constexpr int kBits = 11, kDigits = 1 << kBits, kMaxPasses = (64 + kBits - 1) / kBits;
  const int64_t n = (int64_t)key.size();
  if (n == 0) return;
  const int T = (int)std::max<int64_t>(1, std::min<int64_t>({(int64_t)threads, n / 65536 + 1, 64}));
  auto run = [T](auto &&fn) {  // fn(t) for t in [0, T), on T threads
    std::vector<std::thread> pool;
    std::exception_ptr err[64];
    for (int t = 1; t < T; ++t)
      pool.emplace_back([&, t] {
        try {
          fn(t);
        } catch (...) {
          err[t] = std::current_exception();
        }
      });
    try {
      fn(0);
    } catch (...) {
      err[0] = std::current_exception();
    }
    for (auto &th : pool) th.join();
    for (int t = 0; t < T; ++t)
      if (err[t]) std::rethrow_exception(err[t]);
  };
  auto lo = [n, T](int t) { return n * t / T; };
  // Which digits occur at all: passes beyond the largest key's top digit are
  // skipped.
  std::vector<uint64_t> any_t(T, 0);
  run([&](int t) {
    uint64_t a = 0;
    for (int64_t i = lo(t); i < lo(t + 1); ++i) a |= key[i];
    any_t[t] = a;
  });
  uint64_t any = 0;
  for (uint64_t a : any_t) any |= a;
  int passes = 0;
  while (passes < kMaxPasses && (any >> (passes * kBits)) != 0) ++passes;
  std::vector<uint64_t> key2(n);
  std::vector<int32_t> id2(id ? n : 0);
  std::vector<int64_t> count((size_t)T * kDigits);
  for (int q = 0; q < passes; ++q) {
    const int shift = q * kBits;
    run([&](int t) {
      int64_t *c = count.data() + (size_t)t * kDigits;
      std::fill(c, c + kDigits, 0);
      for (int64_t i = lo(t); i < lo(t + 1); ++i) ++c[(key[i] >> shift) & (kDigits - 1)];
    });
    // One digit value for every key: the order is unchanged.
    bool single = false;
    for (int d = 0; d < kDigits && !single; ++d) {
      int64_t tot = 0;
      for (int t = 0; t < T; ++t) tot += count[(size_t)t * kDigits + d];
      single = tot == n;
    }
    if (single) continue;
    int64_t sum = 0;
    for (int d = 0; d < kDigits; ++d)
      for (int t = 0; t < T; ++t) {
        int64_t &c = count[(size_t)t * kDigits + d];
        const int64_t v = c;
        c = sum;
        sum += v;
      }
    run([&](int t) {
      int64_t *c = count.data() + (size_t)t * kDigits;
      if (id) {
        for (int64_t i = lo(t); i < lo(t + 1); ++i) {
          const int64_t p = c[(key[i] >> shift) & (kDigits - 1)]++;
          key2[p] = key[i];
          id2[p] = (*id)[i];
        }
      } else {
        for (int64_t i = lo(t); i < lo(t + 1); ++i) key2[c[(key[i] >> shift) & (kDigits - 1)]++] = key[i];
      }
    });
    key.swap(key2);
    if (id) id->swap(id2);
  }
}

// Row boundaries of a sorted layout: offsets[k] = first position whose row
// is >= k, for k = 0 .. rows.
static std::vector<int32_t> offsets_of(const std::vector<int32_t> &row, int64_t rows) {
  std::vector<int32_t> off(rows + 1);
  int64_t p = 0;
  const int64_t n = (int64_t)row.size();
  for (int64_t k = 0; k <= rows; ++k) {
    while (p < n && row[p] < k) ++p;
    off[k] = (int32_t)p;
  }
  return off;
}

// Host threads the layout build may use: the hardware's count, at most 16
// (one GPU's share of a host), or KBFOLLOW_HOST_THREADS when set (>= 1).
static int host_threads() {
  if (const char *v = std::getenv("KBFOLLOW_HOST_THREADS")) {
    const int n = std::atoi(v);
    if (n >= 1) return std::min(n, 64);
  }
  const unsigned hw = std::thread::hardware_concurrency();
  return (int)std::max(1u, std::min(hw, 16u));
}

void build_layouts(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                   const int32_t *subj, const int32_t *rel, const int32_t *obj,
                   const float *weight, bool keep_perm, bool keep_offsets, LayoutHost out[3],
                   LayoutSort how) {
  // One 64-bit key per triple and order packs (row, second operand, first
  // operand) as bit fields when 2 * bits(N_E - 1) + bits(N_R - 1) <= 64 (any
  // KB up to 2^27 entities at 2^10 relations); otherwise three chained
  // counting sorts per order.
  auto bits = [](int64_t x) {
    int b = 0;
    while (b < 63 && (int64_t(1) << b) <= x) ++b;
    return b;
  };
  const int be = bits(n_entities - 1), br = bits(n_relations - 1);
  const bool radix = how == LayoutSort::kAuto && 2 * be + br <= 64;
  if (radix && n_triples > 0) {
    // Each order on its own thread (three at a time while their scratch,
    // 16-24 bytes per triple each, stays modest).  The key holds the row,
    // the second and the first operand: they are decoded from the sorted
    // keys, and the triple ids are carried along only for the weights and
    // the permutation.
    const bool need_id = weight != nullptr || keep_perm;
    // Host threads: the three orders run side by side (while their scratch
    // stays modest) and each radix sort splits its passes over its share.
    const int budget = host_threads();
    const bool side_by_side = n_triples <= (int64_t(1) << 27);
    const int sort_threads = side_by_side ? std::max(1, budget / 3) : budget;
    auto one = [&](int which) {
      const int64_t n = n_triples;
      std::vector<uint64_t> key(n);
      // key = major << (bits of middle + bits of minor) | middle << (bits of minor) | minor
      const int32_t *major, *middle, *minor;
      int b_mid;
      int64_t rows;
      if (which == BY_OBJ) {  // (o, r, s): row o, runs of r, A = s
        major = obj, middle = rel, minor = subj, b_mid = br, rows = n_entities;
      } else if (which == BY_SUBJ) {  // (s, r, o): row s, runs of r, A = o
        major = subj, middle = rel, minor = obj, b_mid = br, rows = n_entities;
      } else {  // (r, s, o): row r, runs of s, A = o
        major = rel, middle = subj, minor = obj, b_mid = be, rows = n_relations;
      }
      const int s_mid = be, s_major = be + b_mid;
      for (int64_t l = 0; l < n; ++l)
        key[l] = ((uint64_t)major[l] << s_major) | ((uint64_t)middle[l] << s_mid) |
                 (uint64_t)minor[l];
      std::vector<int32_t> ids;
      if (need_id) {
        ids.resize(n);
        for (int64_t l = 0; l < n; ++l) ids[l] = (int32_t)l;
      }
      radix_sort(key, need_id ? &ids : nullptr, sort_threads);
      LayoutHost &L = out[which];
      L.rows = rows;
      L.row.resize(n);
      L.col_a.resize(n);
      L.col_b.resize(n);
      const uint64_t m_minor = (uint64_t(1) << s_mid) - 1, m_mid = (uint64_t(1) << b_mid) - 1;
      for (int64_t p = 0; p < n; ++p) {
        const uint64_t k = key[p];
        L.col_a[p] = (int32_t)(k & m_minor);
        L.col_b[p] = (int32_t)((k >> s_mid) & m_mid);
        L.row[p] = (int32_t)(k >> s_major);
      }
      std::vector<uint64_t>().swap(key);
      if (weight) {
        L.weight.resize(n);
        for (int64_t p = 0; p < n; ++p) L.weight[p] = weight[ids[p]];
      }
      if (keep_offsets) L.offsets = offsets_of(L.row, rows);
      if (keep_perm) L.perm = std::move(ids);
    };
    const bool parallel = side_by_side;
    if (!parallel) {
      for (int which : {BY_OBJ, BY_SUBJ, BY_REL}) one(which);
      return;
    }
    std::exception_ptr err[3];
    auto guarded = [&](int which) {
      try {
        one(which);
      } catch (...) {
        err[which] = std::current_exception();
      }
    };
    std::thread t_subj(guarded, (int)BY_SUBJ), t_rel(guarded, (int)BY_REL);
    guarded(BY_OBJ);
    t_subj.join();
    t_rel.join();
    for (const auto &e : err)
      if (e) std::rethrow_exception(e);
    return;
  }
  std::vector<int32_t> ident(n_triples), t1, t2, by_subj, by_obj, by_rel, count;
  for (int64_t l = 0; l < n_triples; ++l) ident[l] = (int32_t)l;
  std::vector<int32_t> off_subj, off_obj, off_rel;
  // Least significant key first; every pass is stable.
  // (s, r, o): by subject, relation runs inside a row, objects ascending.
  sort_by_key(obj, n_entities, ident, t1, nullptr, count);
  sort_by_key(rel, n_relations, t1, t2, nullptr, count);
  sort_by_key(subj, n_entities, t2, by_subj, keep_offsets ? &off_subj : nullptr, count);
  // (r, s, o): the (s, r, o) order re-sorted by relation.
  sort_by_key(rel, n_relations, by_subj, by_rel, keep_offsets ? &off_rel : nullptr, count);
  // (o, r, s): by object, relation runs inside a row, subjects ascending.
  sort_by_key(subj, n_entities, ident, t1, nullptr, count);
  sort_by_key(rel, n_relations, t1, t2, nullptr, count);
  sort_by_key(obj, n_entities, t2, by_obj, keep_offsets ? &off_obj : nullptr, count);
  std::vector<int32_t>().swap(ident);
  std::vector<int32_t>().swap(t1);
  std::vector<int32_t>().swap(t2);
  std::vector<int32_t>().swap(count);
  // col_a is gathered for every triple, col_b once per run of equal col_b.
  fill_layout(out[BY_OBJ], n_entities, std::move(by_obj), std::move(off_obj), obj, subj, rel,
              weight, keep_perm);
  fill_layout(out[BY_SUBJ], n_entities, std::move(by_subj), std::move(off_subj), subj, obj, rel,
              weight, keep_perm);
  fill_layout(out[BY_REL], n_relations, std::move(by_rel), std::move(off_rel), rel, obj, subj,
              weight, keep_perm);
}

// Rows [first, first + count) as pieces of at most kEmptyPiece rows.
static void add_empty(PlanHost &P, int64_t first, int64_t count) {
  P.n_empty_rows += count;
  for (int64_t q = first; q < first + count; q += kEmptyPiece)
    P.empty.push_back({(int32_t)q, (int32_t)std::min<int64_t>(kEmptyPiece, first + count - q)});
}

// Classes of the gathered ids, about equal in the number of triples that
// gather each: the heaviest ids one by one onto the lightest class, the
// others by id modulo n_xcd.  Empty when the id space is far larger than the
// KB (then the class of id a is a % n_xcd).
static std::vector<uint8_t> id_classes(const std::vector<int32_t> &col, int64_t n_ids, int X) {
  const int64_t n_t = (int64_t)col.size();
  if (X <= 1 || n_ids <= 0 || n_ids > 4 * n_t + (int64_t(1) << 20)) return {};
  std::vector<int32_t> cnt(n_ids, 0);
  for (int32_t a : col) ++cnt[a];
  std::vector<uint8_t> cls(n_ids);
  const int64_t k_heavy = std::min<int64_t>(n_ids, 65536);
  // The k_heavy heaviest ids (ties to the smaller id), heaviest first: the
  // count of the k-th one from a selection, then the ids above it and as
  // many of those at it as are needed, in id order.
  std::vector<int32_t> heavy;
  if (k_heavy > 0) {
    std::vector<int32_t> c(cnt);
    std::nth_element(c.begin(), c.begin() + (k_heavy - 1), c.end(), std::greater<int32_t>());
    const int32_t kth = c[k_heavy - 1];
    std::vector<int32_t>().swap(c);
    int64_t above = 0;
    for (int64_t i = 0; i < n_ids; ++i) above += cnt[i] > kth;
    int64_t at_kth = k_heavy - above;
    heavy.reserve(k_heavy);
    for (int64_t i = 0; i < n_ids; ++i)
      if (cnt[i] > kth || (cnt[i] == kth && at_kth-- > 0)) heavy.push_back((int32_t)i);
    std::sort(heavy.begin(), heavy.end(),
              [&](int32_t x, int32_t y) { return cnt[x] != cnt[y] ? cnt[x] > cnt[y] : x < y; });
  }
  std::vector<char> is_heavy(n_ids, 0);
  for (int32_t h : heavy) is_heavy[h] = 1;
  int64_t load[kMaxXcd] = {};
  for (int64_t i = 0; i < n_ids; ++i)
    if (!is_heavy[i]) {
      cls[i] = (uint8_t)(i % X);
      load[i % X] += cnt[i];
    }
  for (int32_t h : heavy) {
    int best = 0;
    for (int k = 1; k < X; ++k)
      if (load[k] < load[best]) best = k;
    cls[h] = (uint8_t)best;
    load[best] += cnt[h];
  }
  return cls;
}

double top_id_share(const std::vector<int32_t> &col, int64_t n_ids, double frac) {
  if (col.empty() || n_ids <= 0) return 0.0;
  std::vector<int32_t> cnt((size_t)n_ids, 0);
  for (int32_t id : col) ++cnt[(size_t)id];
  const int64_t k = std::min<int64_t>(
      n_ids, std::max<int64_t>(1, (int64_t)std::ceil(frac * (double)n_ids)));
  if (k < n_ids) std::nth_element(cnt.begin(), cnt.begin() + k, cnt.end(), std::greater<int32_t>());
  int64_t top = 0;
  for (int64_t i = 0; i < k; ++i) top += cnt[(size_t)i];
  return (double)top / (double)col.size();
}

PlanHost plan_layout(const LayoutHost &L, int32_t chunk, int32_t fan_in) {
  PlanOptions o;
  o.chunk = chunk;
  o.fan_in = fan_in;
  o.n_xcd = 1;
  return plan_layout(L, o);
}

PlanHost plan_layout(const LayoutHost &L, const PlanOptions &opt) {
  PlanHost P;
  const int32_t chunk = opt.chunk, fan_in = opt.fan_in;
  const int X = std::max(1, std::min<int>(opt.n_xcd, kMaxXcd));
  P.chunk = chunk;
  P.fan_in = fan_in;
  P.n_xcd = X;
  const bool weighted = !L.weight.empty();
  const int64_t n_t = (int64_t)L.col_a.size();

  // Rows with triples, in row order; the rows between them are empty.
  struct RowSpan {
    int32_t row;
    int64_t beg, end;
  };
  std::vector<RowSpan> rows;
  int64_t next_row = 0;
  for (int64_t beg = 0, end; beg < n_t; beg = end) {
    const int32_t q = L.row[beg];
    for (end = beg + 1; end < n_t && L.row[end] == q;) ++end;
    add_empty(P, next_row, q - next_row);
    next_row = (int64_t)q + 1;
    P.max_row_len = std::max(P.max_row_len, end - beg);
    rows.push_back({q, beg, end});
  }
  add_empty(P, next_row, L.rows - next_row);

  // The order in which triples enter the stream: the layout's own, except
  // inside hub rows of a plan with several lists.
  std::vector<int32_t> pos(n_t);
  for (int64_t i = 0; i < n_t; ++i) pos[i] = (int32_t)i;
  const std::vector<int32_t> &cls_col = opt.class_by_b ? L.col_b : L.col_a;
  const std::vector<uint8_t> cls_tab =
      id_classes(cls_col, opt.class_by_b ? opt.n_ids_b : opt.n_ids_a, X);
  // The class of the triple at position l.
  auto cls_at = [&](int64_t l) -> int {
    const int32_t id = cls_col[l];
    return cls_tab.empty() ? (int)(id % X) : (int)cls_tab[id];
  };

  // Segments per list: a hub row's class segments first (rows in order),
  // then whole rows.  `alone`: the segment is its row's only one.
  struct Seg {
    int32_t row;
    int64_t beg, end;  // into pos
    bool alone, hub;
  };
  std::vector<std::vector<Seg>> segs(X);
  if (X == 1) {
    for (const RowSpan &r : rows) segs[0].push_back({r.row, r.beg, r.end, true, false});
  } else {
    int64_t load[kMaxXcd] = {};
    std::vector<uint64_t> key;
    std::vector<int32_t> idx;
    std::vector<std::pair<uint64_t, int32_t>> kp;
    const int sort_threads = std::max(1, host_threads() / 3);
    const int32_t a_blocks =
        opt.hub_by_a ? 0 : std::max<int32_t>(0, std::min<int32_t>(opt.a_blocks, 64));
    std::vector<const RowSpan *> small;
    int64_t total = 0;
    for (const RowSpan &r : rows) {
      const int64_t len = r.end - r.beg;
      total += len + 1;
      if (len < opt.hub_min) {
        small.push_back(&r);
        continue;
      }
      // (class, gathered id, second operand) or (class, second operand,
      // gathered id) as one 64-bit key per triple, the ids in as many bits
      // as the row's largest needs (at most 3 + 30 + 30), sorted stably:
      // long rows by the radix sort, others as (key, position) pairs.
      uint64_t mx = 0, my = 0;
      for (int64_t l = r.beg; l < r.end; ++l) {
        mx = std::max<uint64_t>(mx, (uint64_t)(opt.hub_by_a ? L.col_a[l] : L.col_b[l]));
        my = std::max<uint64_t>(my, (uint64_t)(opt.hub_by_a ? L.col_b[l] : L.col_a[l]));
      }
      int bx = 0, by = 0;
      while (bx < 63 && (mx >> bx) != 0) ++bx;
      while (by < 63 && (my >> by) != 0) ++by;
      // Blocks of the gathered id ahead of the second operand (3 bits of
      // class, at most 6 of block).
      int bk = 0;
      if (a_blocks > 1) {
        while ((1 << bk) < a_blocks) ++bk;
        if (3 + bk + bx + by > 64) bk = 0;
      }
      auto key_of = [&](int64_t l) {
        const uint64_t c = (uint64_t)cls_at(l);
        const uint64_t x = (uint64_t)(opt.hub_by_a ? L.col_a[l] : L.col_b[l]);
        const uint64_t y = (uint64_t)(opt.hub_by_a ? L.col_b[l] : L.col_a[l]);
        const uint64_t k =
            bk ? (uint64_t)((int64_t)L.col_a[l] * a_blocks / std::max<int64_t>(1, opt.n_ids_a))
               : 0;
        return (c << (bk + bx + by)) | (k << (bx + by)) | (x << by) | y;
      };
      if (len >= (int64_t(1) << 16)) {
        key.resize(len);
        idx.resize(len);
        for (int64_t i = 0; i < len; ++i) {
          key[i] = key_of(r.beg + i);
          idx[i] = (int32_t)i;
        }
        radix_sort(key, &idx, sort_threads);
        for (int64_t i = 0; i < len; ++i) pos[r.beg + i] = (int32_t)(r.beg + idx[i]);
      } else {
        kp.resize(len);
        for (int64_t i = 0; i < len; ++i) kp[i] = {key_of(r.beg + i), (int32_t)i};
        std::sort(kp.begin(), kp.end());
        for (int64_t i = 0; i < len; ++i) pos[r.beg + i] = (int32_t)(r.beg + kp[i].second);
      }
      // One segment per class present.
      std::vector<Seg> mine;
      for (int64_t b0 = r.beg, b1; b0 < r.end; b0 = b1) {
        const int c = cls_at(pos[b0]);
        for (b1 = b0 + 1; b1 < r.end && cls_at(pos[b1]) == c;) ++b1;
        mine.push_back({r.row, b0, b1, false, true});
        load[c] += b1 - b0 + 1;
      }
      const bool alone = mine.size() == 1;
      for (Seg &g : mine) {
        g.alone = alone;
        segs[cls_at(pos[g.beg])].push_back(g);
      }
    }
    // Whole rows: the list of their first gathered id's class while it has
    // room, else the lightest list, so that every list gets about the same
    // number of entries.
    const int64_t target = (total + X - 1) / X;
    for (const RowSpan *r : small) {
      const int64_t w = r->end - r->beg + 1;
      int c = cls_at(r->beg);
      if (load[c] + w > target) {
        for (int k = 0; k < X; ++k)
          if (load[k] < load[c]) c = k;
      }
      segs[c].push_back({r->row, r->beg, r->end, true, false});
      load[c] += w;
    }
  }

  // Each list's stream.  A marker that writes a partial sum gets a pending
  // slot (row, list, index within the segment's partials); slots are
  // numbered once every list is built, consecutively per row.
  struct Pend {
    int32_t row, list, idx;
    int64_t at;  // entry within its list's stream
  };
  std::vector<Pend> pend;
  std::vector<std::vector<Entry>> S(X);
  std::vector<std::vector<float>> Wt(X);
  std::vector<std::vector<int32_t>> first_a(X);  // per chunk: first gathered id, or -1
  std::vector<std::vector<char>> hub_chunk(X);   // per chunk: starts inside a hub segment
  for (int x = 0; x < X; ++x) {
    std::vector<Entry> &E = S[x];
    std::vector<float> &Wv = Wt[x];
    int64_t est = 0;
    for (const Seg &g : segs[x]) est += g.end - g.beg + 1;
    E.reserve(est + est / std::max(1, chunk - 1) + chunk + 2);
    auto marker = [&](int32_t target) {
      E.push_back({kMarker, target});
      if (weighted) Wv.push_back(0.0f);
    };
    auto slot_marker = [&](int32_t row, int32_t idx) {
      pend.push_back({row, x, idx, (int64_t)E.size()});
      marker(kNoTarget);  // target set when the slots are numbered
    };
    for (const Seg &g : segs[x]) {
      int32_t parts = 0;
      bool pending = false;  // triples of this segment since the last marker
      int32_t prev_b = 0, prev_a = -1;
      for (int64_t p = g.beg; p < g.end; ++p) {
        if ((int64_t)E.size() % chunk == chunk - 1) {
          // The chunk's last entry must be a marker.
          if (pending)
            slot_marker(g.row, parts++);
          else
            marker(kNoTarget);
          pending = false;
        }
        const int32_t l = pos[p];
        // A run starts after every marker and wherever col_b changes.
        const bool run_start = !pending || L.col_b[l] != prev_b;
        // The previous entry (a triple of this row, not across a step
        // boundary) gathered the same row: the kernel reuses it.
        const bool same_a = pending && L.col_a[l] == prev_a &&
                            (int64_t)E.size() % kStepEntries != 0;
        const int64_t c = (int64_t)E.size() / chunk;
        if ((int64_t)first_a[x].size() <= c) {
          first_a[x].resize(c + 1, -1);
          hub_chunk[x].resize(c + 1, 0);
        }
        if (first_a[x][c] < 0) {
          first_a[x][c] = L.col_a[l];
          hub_chunk[x][c] = g.hub;
        }
        E.push_back({L.col_a[l] | (run_start ? kRunStart : 0), L.col_b[l] | (same_a ? kSameA : 0)});
        if (weighted) Wv.push_back(L.weight[l]);
        prev_b = L.col_b[l];
        prev_a = L.col_a[l];
        pending = true;
      }
      if (!g.alone || parts > 0)
        slot_marker(g.row, parts++);
      else
        marker(g.row);
    }
    // Pad with no-op markers to whole chunks: every lane group then walks
    // exactly `chunk` entries.
    while ((int64_t)E.size() % chunk != 0) marker(kNoTarget);
    first_a[x].resize(E.size() / chunk, -1);
    hub_chunk[x].resize(E.size() / chunk, 0);
  }

  // Slots: per row in (list, index) order, rows in row order.
  std::vector<int32_t> order(pend.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (int32_t)i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t u, int32_t v) {
    const Pend &a = pend[u], &b = pend[v];
    if (a.row != b.row) return a.row < b.row;
    if (a.list != b.list) return a.list < b.list;
    return a.idx < b.idx;
  });
  struct Split {
    int32_t row;
    int64_t first, n;
  };
  std::vector<Split> splits;
  for (size_t i = 0; i < order.size();) {
    const int32_t row = pend[order[i]].row;
    const int64_t first = P.n_slots;
    size_t j = i;
    for (; j < order.size() && pend[order[j]].row == row; ++j) {
      const Pend &q = pend[order[j]];
      S[q.list][q.at].y = -(int32_t)P.n_slots - 1;
      ++P.n_slots;
    }
    splits.push_back({row, first, (int64_t)(j - i)});
    ++P.n_split_rows;
    i = j;
  }

  // Chunk order inside each list: hub chunks by their first gathered id,
  // then the others in stream order.
  P.xcd_chunk.assign(1, 0);
  {
    size_t total_entries = 0;
    for (int x = 0; x < X; ++x) total_entries += S[x].size();
    P.entries.reserve(total_entries);
    if (weighted) P.weights.reserve(total_entries);
  }
  for (int x = 0; x < X; ++x) {
    const int64_t nc = (int64_t)S[x].size() / chunk;
    std::vector<int64_t> co(nc);
    for (int64_t c = 0; c < nc; ++c) co[c] = c;
    if (X > 1 && opt.band)
      std::stable_sort(co.begin(), co.end(), [&](int64_t u, int64_t v) {
        const bool hu = hub_chunk[x][u], hv = hub_chunk[x][v];
        if (hu != hv) return hu;
        return hu && first_a[x][u] < first_a[x][v];
      });
    for (int64_t c : co) {
      P.entries.insert(P.entries.end(), S[x].begin() + c * chunk, S[x].begin() + (c + 1) * chunk);
      if (weighted)
        P.weights.insert(P.weights.end(), Wt[x].begin() + c * chunk,
                         Wt[x].begin() + (c + 1) * chunk);
    }
    std::vector<Entry>().swap(S[x]);
    std::vector<float>().swap(Wt[x]);
    P.xcd_chunk.push_back((int64_t)P.entries.size() / chunk);
  }
  P.n_chunks = (int64_t)P.entries.size() / chunk;

  // Combine levels: a row split into n partials is reduced fan_in slots at a
  // time until one task writes the row.
  for (const Split &sp : splits) {
    int64_t first_slot = sp.first, cnt = sp.n;
    size_t level = 0;
    while (cnt > fan_in) {
      const int64_t groups = (cnt + fan_in - 1) / fan_in;
      const int64_t out0 = P.n_slots;
      P.n_slots += groups;
      if (P.levels.size() <= level) P.levels.resize(level + 1);
      for (int64_t g = 0; g < groups; ++g) {
        const int64_t m = std::min<int64_t>(fan_in, cnt - g * fan_in);
        P.levels[level].push_back({(int32_t)(first_slot + g * fan_in), (int32_t)m,
                                   (int32_t)(-(out0 + g) - 1), 0});
      }
      first_slot = out0;
      cnt = groups;
      ++level;
    }
    if (P.levels.size() <= level) P.levels.resize(level + 1);
    P.levels[level].push_back({(int32_t)first_slot, (int32_t)cnt, sp.row, 0});
  }
  return P;
}

}  // namespace kbf
