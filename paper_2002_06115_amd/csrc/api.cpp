// api.cpp -- the C ABI of kbfollow.h: KB construction, the three passes,
// workspace sizing, errors and event-based kernel timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <exception>
#include <initializer_list>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <utility>
#include <vector>

#include "kbfollow.h"
#include "kernels.h"
#include "plan.h"

using namespace kbf;

namespace {

thread_local std::string g_last_error;

kb_status fail(kb_status s, const std::string &msg) {
  g_last_error = msg;
  return s;
}

kb_status hip_fail(hipError_t e, const char *what) {
  return fail(KB_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Stream plan of one layout, resident on the device.
struct DevLayout {
  int64_t rows = 0;
  int2 *entries = nullptr;    // the entry stream (triples and markers)
  float *weights = nullptr;   // per entry, soft KB only
  int64_t n = 0;
  int32_t chunk = 0;
  int64_t n_chunks = 0;
  int2 *empty = nullptr;      // pieces (first row, count) of rows no triple reaches
  int64_t n_empty_pieces = 0;
  int64_t n_empty = 0;        // rows in those pieces
  int4 *ctasks = nullptr;     // all combine levels, back to back
  std::vector<int64_t> level_begin;  // host: level L is [level_begin[L], level_begin[L+1])
  int64_t n_slots = 0;
  int64_t n_split_rows = 0;
  int64_t max_row_len = 0;
  int32_t n_lists = 1;                 // chunk lists, one per XCD
  int64_t list_chunk[kMaxChunkLists + 1] = {};
};

struct Timing {
  uint32_t mask = 0;  // bit p set: phase p is recorded
  std::vector<hipEvent_t> pool;
  struct Rec {
    int phase;
    hipEvent_t start, stop;
  };
  std::vector<Rec> recs;
};

int env_int(const char *name, int dflt) {
  const char *v = std::getenv(name);
  if (!v || !*v) return dflt;
  return std::atoi(v);
}

}  // namespace

struct kb_t {
  int device = 0;
  int n_cu = 0;
  int64_t n_entities = 0, n_relations = 0, n_triples = 0;
  bool weighted = false;
  bool plain_loads = false;  // force plain loads instead of raw buffer loads (testing)
  bool b_in_lds = true;      // stage small B tables in LDS (off: B rows in registers)
  bool stream_stamps = true; // time stream kernels by their dispatch timestamps (off: event records)
  int max_lpt = 0;           // widest lane group of the register variant; 0: per pass (lane_cap)
  // The backward's dR pass on a stream of the KB's own, concurrent with the
  // dX pass: -1 on large KBs at b <= 32, 1 always, 0 never; the stream, fork
  // and join events, and a lock that keeps one call's record / wait
  // sequence whole when threads share the KB (side is null when never).
  int overlap_backward = 0;
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  mutable std::mutex side_mu;
  DevLayout L[3];
  std::vector<void *> allocations;
  int64_t device_bytes = 0;
  mutable Timing timing;
};

namespace {

// Copies n elements of `host` into a new device allocation owned by the KB.
template <class T, class D>
kb_status upload(kb_t *kb, const T *host, size_t n, D **dev, hipStream_t s) {
  static_assert(sizeof(T) == sizeof(D), "same element layout on both sides");
  *dev = nullptr;
  if (n == 0) return KB_OK;
  const size_t bytes = n * sizeof(T);
  void *p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(KB_ENOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  kb->allocations.push_back(p);
  kb->device_bytes += (int64_t)bytes;
  e = hipMemcpyAsync(p, host, bytes, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  *dev = static_cast<D *>(p);
  return KB_OK;
}

template <class T, class D>
kb_status upload(kb_t *kb, const std::vector<T> &host, D **dev, hipStream_t s) {
  return upload(kb, host.data(), host.size(), dev, s);
}

void free_kb(kb_t *kb) {
  if (kb->side) (void)hipStreamDestroy(kb->side);
  if (kb->ev_fork) (void)hipEventDestroy(kb->ev_fork);
  if (kb->ev_join) (void)hipEventDestroy(kb->ev_join);
  for (void *p : kb->allocations) (void)hipFree(p);
  for (hipEvent_t ev : kb->timing.pool) (void)hipEventDestroy(ev);
  for (auto &r : kb->timing.recs) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  delete kb;
}

// Uploads one layout's stream plan (made by plan_layout from its sorted
// rows) and waits for the copies.
kb_status build_device_layout(kb_t *kb, DevLayout &D, int64_t rows, const PlanHost &P,
                              int32_t chunk, hipStream_t s) {
  D.rows = rows;
  D.n = (int64_t)P.entries.size();
  D.chunk = chunk;
  D.n_chunks = P.n_chunks;
  D.n_empty = P.n_empty_rows;
  D.n_empty_pieces = (int64_t)P.empty.size();
  D.n_slots = P.n_slots;
  D.n_split_rows = P.n_split_rows;
  D.max_row_len = P.max_row_len;
  static_assert(kMaxXcd == kMaxChunkLists, "one chunk list per XCD");
  D.n_lists = P.n_xcd;
  for (int x = 0; x <= P.n_xcd; ++x) D.list_chunk[x] = P.xcd_chunk[x];
  static_assert(sizeof(Entry) == sizeof(int2), "entry layout");
  static_assert(sizeof(EmptyPiece) == sizeof(int2), "empty-piece layout");
  std::vector<int4> ctasks;
  D.level_begin.assign(1, 0);
  for (const auto &lv : P.levels) {
    for (const CombineTask &c : lv) ctasks.push_back(make_int4(c.first, c.n, c.dst, 0));
    D.level_begin.push_back((int64_t)ctasks.size());
  }
  kb_status st;
  if ((st = upload(kb, P.entries, &D.entries, s)) != KB_OK) return st;
  if ((st = upload(kb, P.weights, &D.weights, s)) != KB_OK) return st;
  if ((st = upload(kb, P.empty, &D.empty, s)) != KB_OK) return st;
  if ((st = upload(kb, ctasks, &D.ctasks, s)) != KB_OK) return st;
  // The host vectors may die after this call: wait for the copies first.
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  return KB_OK;
}

// Event bracket around one phase's launches.
struct PhaseScope {
  const kb_t *kb;
  int phase;
  hipStream_t s;
  hipEvent_t start = nullptr, stop = nullptr;
  static hipEvent_t take(Timing &t) {
    if (!t.pool.empty()) {
      hipEvent_t e = t.pool.back();
      t.pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  // record_events: record start now and stop at the end of the scope;
  // otherwise the events go to the scope's one kernel launch, which sets
  // them (see launch_stream), and the scope only files them.
  bool record_events = true;
  PhaseScope(const kb_t *k, int ph, hipStream_t st, bool record = true)
      : kb(k), phase(ph), s(st), record_events(record) {
    if (!((kb->timing.mask >> phase) & 1u)) return;
    start = take(kb->timing);
    stop = take(kb->timing);
    if (start && stop && record_events) (void)hipEventRecord(start, s);
  }
  // The events to hand to the scope's kernel launch (null when not timed).
  hipEvent_t launch_start() const { return (start && stop && !record_events) ? start : nullptr; }
  hipEvent_t launch_stop() const { return (start && stop && !record_events) ? stop : nullptr; }
  ~PhaseScope() {
    if (start && stop) {
      if (record_events) (void)hipEventRecord(stop, s);
      kb->timing.recs.push_back({phase, start, stop});
      return;
    }
    // Only one event could be created: keep it for later, record nothing.
    if (start) kb->timing.pool.push_back(start);
    if (stop) kb->timing.pool.push_back(stop);
  }
};

bool overlaps(const void *a, size_t abytes, const void *b, size_t bbytes) {
  if (!a || !b || !abytes || !bbytes) return false;
  const char *pa = static_cast<const char *>(a), *pb = static_cast<const char *>(b);
  return pa < pb + bbytes && pb < pa + abytes;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

kb_status check_device(const kb_t *kb) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != kb->device)
    return fail(KB_EINVAL, "the current HIP device is " + std::to_string(dev) +
                               " but the KB lives on device " + std::to_string(kb->device));
  return KB_OK;
}

// The widest lane group of the register variant for a pass.  Narrower lane
// groups mean more column slices, each gathering from a narrower part of the
// table and re-reading the entry stream.  That pays for the dR pass (B = X,
// read in registers) at b >= 128: 32-column slices took the training-shaped
// KB's dR from 3.92 to 3.80 ms at b = 256, the 10 M-entity KB's from 3.51 to
// 3.42 ms at b = 128 and the MetaQA-shaped KB's from 0.0182 to 0.0175 ms,
// while at b = 64 they cost 1 % and the forward and dX register variants at
// b = 128 and 256 lost 12-15 %.
int lane_cap(const kb_t *kb, int ph_base, int32_t b) {
  if (kb->max_lpt > 0) return kb->max_lpt;
  return (ph_base == KB_PH_DR_STREAM && b >= 128) ? 8 : 32;
}

// Runs one pass: the stream kernel, the first combine level together with
// the empty rows, the further combine levels.  With Z non-null (one row per
// output row; A itself for the residual hop, out itself to add in place)
// every output row j also gets gamma * Z[j].
kb_status run_pass(const kb_t *kb, const DevLayout &D, int ph_base, const float *A,
                   int64_t A_rows, const float *B, int64_t B_rows, int32_t b, float *out,
                   void *ws, const float *Z, float gamma, hipStream_t s) {
  double *slots = static_cast<double *>(ws);
  const float *res = Z;
  if (D.n > 0) {
    // Timed by the kernel's own timestamps: no event packets between this
    // launch and the next, which would hold back a concurrent pass.
    PhaseScope scope(kb, ph_base + 0, s, !kb->stream_stamps);
    StreamArgs a{D.entries, D.weights, D.n, D.chunk, A,           A_rows,     B,
                 B_rows,    b,         out,  D.rows,  slots, D.n_slots, Z ? 1 : 0, gamma, Z,
                 D.n_lists, {}};
    std::copy(D.list_chunk, D.list_chunk + kMaxChunkLists + 1, a.list_chunk);
    StreamOptions o;
    o.plain_loads = kb->plain_loads;
    o.b_in_lds = kb->b_in_lds;
    o.n_cu = kb->n_cu;
    o.max_lpt = lane_cap(kb, ph_base, b);
    hipError_t e = launch_stream(a, o, s, scope.launch_start(), scope.launch_stop());
    if (e != hipSuccess) return hip_fail(e, "stream kernel launch");
  }
  {
    // The first combine level and the empty rows share one launch.
    PhaseScope scope(kb, ph_base + 1, s);
    const int64_t n0 = D.level_begin.size() > 1 ? D.level_begin[1] - D.level_begin[0] : 0;
    TailArgs t{D.ctasks, n0, slots, D.n_slots, D.empty, D.n_empty_pieces, b, out, D.rows, res,
               gamma, 0};
    hipError_t e = launch_tail(t, s);
    if (e != hipSuccess) return hip_fail(e, "combine and empty-row kernel launch");
  }
  {
    PhaseScope scope(kb, ph_base + 2, s);
    for (size_t L = 1; L + 1 < D.level_begin.size(); ++L) {
      const int64_t n = D.level_begin[L + 1] - D.level_begin[L];
      hipError_t e = launch_combine(D.ctasks + D.level_begin[L], n, slots, D.n_slots, b, out,
                                    D.rows, res, gamma, s);
      if (e != hipSuccess) return hip_fail(e, "combine kernel launch");
    }
  }
  return KB_OK;
}

size_t round256(size_t x) { return (x + 255) / 256 * 256; }

// Byte offset of the dR pass's slots in the workspace: after the dX pass's,
// so that the two passes can run concurrently.
size_t dr_slots_offset(const kb_t *kb, int32_t b) {
  return round256((size_t)kb->L[BY_SUBJ].n_slots * (size_t)b * sizeof(double));
}

size_t workspace_bytes(const kb_t *kb, int32_t b) {
  const size_t fwd = round256((size_t)kb->L[BY_OBJ].n_slots * (size_t)b * sizeof(double));
  const size_t bwd = dr_slots_offset(kb, b) +
                     round256((size_t)kb->L[BY_REL].n_slots * (size_t)b * sizeof(double));
  return std::max(fwd, bwd);
}

// The workspace must be big enough, aligned, and clear of every array the
// call reads or writes (arrays[i] of bytes[i]; null entries are skipped).
kb_status check_ws(const kb_t *kb, int32_t b, void *ws, size_t ws_bytes,
                   std::initializer_list<std::pair<const void *, size_t>> arrays) {
  const size_t need = workspace_bytes(kb, b);
  if (need == 0) return KB_OK;
  if (!ws) return fail(KB_EINVAL, "workspace is NULL but " + std::to_string(need) + " bytes are needed");
  if (ws_bytes < need)
    return fail(KB_EINVAL, "workspace has " + std::to_string(ws_bytes) + " bytes, " +
                               std::to_string(need) + " are needed");
  if (!aligned(ws, 16)) return fail(KB_EINVAL, "workspace must be 16-byte aligned");
  for (const auto &a : arrays)
    if (overlaps(ws, need, a.first, a.second))
      return fail(KB_EINVAL, "workspace overlaps an input or output array");
  return KB_OK;
}

}  // namespace

extern "C" {

const char *kb_status_str(kb_status s) {
  switch (s) {
    case KB_OK: return "ok";
    case KB_EINVAL: return "invalid argument";
    case KB_ERANGE: return "id out of range";
    case KB_ENOMEM: return "out of memory";
    case KB_EHIP: return "HIP runtime error";
    case KB_ENOTSUP: return "not supported";
  }
  return "unknown status";
}

const char *kb_last_error(void) { return g_last_error.c_str(); }

kb_status kb_layout_host(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                         const int32_t *subj, const int32_t *rel, const int32_t *obj,
                         int32_t which, int32_t *offsets, int32_t *col_a, int32_t *col_b,
                         int32_t *perm) {
  try {
    g_last_error.clear();
    if (which < 0 || which > 2) return fail(KB_EINVAL, "which must be 0, 1 or 2");
    bool range = false;
    std::string msg = validate_triples(n_entities, n_relations, n_triples, subj, rel, obj, &range);
    if (!msg.empty()) return fail(range ? KB_ERANGE : KB_EINVAL, msg);
    LayoutHost L[3];
    build_layouts(n_entities, n_relations, n_triples, subj, rel, obj, nullptr, true, true, L);
    const LayoutHost &H = L[which];
    if (offsets) std::copy(H.offsets.begin(), H.offsets.end(), offsets);
    if (col_a) std::copy(H.col_a.begin(), H.col_a.end(), col_a);
    if (col_b) std::copy(H.col_b.begin(), H.col_b.end(), col_b);
    if (perm) std::copy(H.perm.begin(), H.perm.end(), perm);
    return KB_OK;
  } catch (const std::bad_alloc &) {
    return fail(KB_ENOMEM, "host allocation failed");
  } catch (...) {
    return fail(KB_EINVAL, "unexpected host error");
  }
}

kb_status kb_create(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                    const int32_t *subj, const int32_t *rel, const int32_t *obj,
                    const float *weight, void *stream, kb_t **out) {
  if (!out) return fail(KB_EINVAL, "out must be non-NULL");
  *out = nullptr;
  kb_t *kb = nullptr;
  try {
    g_last_error.clear();
    bool range = false;
    std::string msg = validate_triples(n_entities, n_relations, n_triples, subj, rel, obj, &range);
    if (!msg.empty()) return fail(range ? KB_ERANGE : KB_EINVAL, msg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    kb = new kb_t();
    hipError_t e = hipGetDevice(&kb->device);
    if (e != hipSuccess) {
      free_kb(kb);
      return hip_fail(e, "hipGetDevice");
    }
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, kb->device) == hipSuccess)
      kb->n_cu = v;
    if (kb->n_cu <= 0) kb->n_cu = 1;
    kb->plain_loads = env_int("KBFOLLOW_PLAIN_LOADS", 0) != 0;
    kb->b_in_lds = env_int("KBFOLLOW_B_IN_LDS", 1) != 0;
    kb->stream_stamps = env_int("KBFOLLOW_STREAM_STAMPS", 1) != 0;
    kb->max_lpt = env_int("KBFOLLOW_MAX_LPT", 0);
    // dR concurrent with dX from 2^20 triples on, at b <= 32 (measured on the
    // large KB: steps 3-5 % shorter at b = 8 .. 32, 4 % longer at b = 64, the
    // same at 128 and 256; on small KBs the fork and join cost more than
    // they save).
    {
      const int forced = env_int("KBFOLLOW_OVERLAP_BACKWARD", -1);
      kb->overlap_backward = forced >= 0 ? (forced != 0 ? 1 : 0)
                                         : (n_triples >= (int64_t(1) << 20) ? -1 : 0);
    }
    if (kb->overlap_backward != 0) {
      hipError_t e2 = hipStreamCreateWithFlags(&kb->side, hipStreamNonBlocking);
      if (e2 == hipSuccess) e2 = hipEventCreateWithFlags(&kb->ev_fork, hipEventDisableTiming);
      if (e2 == hipSuccess) e2 = hipEventCreateWithFlags(&kb->ev_join, hipEventDisableTiming);
      if (e2 != hipSuccess) {
        free_kb(kb);
        return hip_fail(e2, "stream and events of the concurrent backward");
      }
    }
    kb->n_entities = n_entities;
    kb->n_relations = n_relations;
    kb->n_triples = n_triples;
    kb->weighted = weight != nullptr;
    // Chunk length: 256 entries, shorter for small streams so that there are
    // at least ~32 K chunks to spread over the GPU (never below 16).
    auto default_chunk = [](int64_t entries) {
      int32_t c = 256;
      while (c > 16 && entries / c < 32768) c /= 2;
      return c;
    };
    // A chunk is a whole number of kernel steps.
    auto whole_steps = [](int32_t c) {
      return std::max(kChunkQuantum, (c + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum);
    };
    const int32_t chunk_seg =
        whole_steps(env_int("KBFOLLOW_CHUNK", default_chunk(n_triples + n_entities)));
    // dR's chunks at most 128 entries: with its object blocks, the shorter
    // chunks keep the gathers in flight at once closer together (measured on
    // one box: 10 M-entity KB step 2.369 -> 2.340 ms, training-shaped KB
    // 9.05 -> 9.00 ms; 64 no better), for twice the partial slots.
    const int32_t chunk_rel = whole_steps(env_int(
        "KBFOLLOW_REL_CHUNK", std::min<int32_t>(128, default_chunk(n_triples + n_relations))));
    const int32_t fan_in = std::max(2, env_int("KBFOLLOW_FAN_IN", 32));
    {
      LayoutHost H[3];
      const char *how = std::getenv("KBFOLLOW_LAYOUT_SORT");
      build_layouts(n_entities, n_relations, n_triples, subj, rel, obj, weight, false, false, H,
                    how && std::strcmp(how, "counting") == 0 ? LayoutSort::kCounting
                                                             : LayoutSort::kAuto);
      // The three plans on three host threads, then the uploads in turn.
      const int32_t plen[3] = {chunk_seg, chunk_seg, chunk_rel};
      // One chunk list per XCD (8 on an MI355X; KBFOLLOW_XCD overrides, 1 is
      // a single list in row order).  Hub rows (KBFOLLOW_HUB_MIN triples or
      // more) are split by the class of the gathered id; in the forward and
      // dX passes (second operand R, read from LDS) their triples are ordered
      // by gathered id, in the dR pass by (object block, subject, object),
      // which keeps runs of equal subject, whose X row is read once per run.
      const int32_t n_xcd = std::max(1, std::min(kMaxXcd, env_int("KBFOLLOW_XCD", 8)));
      const int64_t hub_min = std::max(1, env_int("KBFOLLOW_HUB_MIN", 256));
      const bool band = env_int("KBFOLLOW_BAND", 1) != 0;
      // dR's lists are classed by subject (the X row read once per run) when
      // the objects are skewed, by the gathered object when they are not
      // (KBFOLLOW_DR_CLASS_B=1 / 0 forces one).  Skewed objects (the top 1 %
      // by in-degree holding at least a quarter of the triples) keep their
      // dY rows hot in the L2s under any classing, and subject classes keep
      // every (relation, subject) run whole: on the 10 M-entity KB (top 1 %
      // of the Zipf objects: ~80 % of the triples) dR took 0.797 ms with
      // object classes and 0.775 with subject classes (passes serial; 3.21
      // against 3.11 ms at b = 128, 6.51 against 6.27 at b = 256).  With
      // near-uniform objects only the classing keeps one XCD's dY working
      // set small: on the training-shaped KB (uniform objects) dR took 3.04
      // ms with object classes and 3.45 with subject classes (64 blocks
      // each; 0.391 against 0.439 ms at b = 32).
      const int cls_env = env_int("KBFOLLOW_DR_CLASS_B", -1);
      const bool dr_class_b = cls_env >= 0
                                  ? cls_env != 0
                                  : top_id_share(H[BY_REL].col_a, n_entities, 0.01) >= 0.25;
      // dR's hub segments led by 64 blocks of the object id, so that the
      // chunks in flight at once gather dY from a few blocks: dR 0.815 ->
      // 0.79 ms on the 10 M-entity KB with the passes serial (8 to 32 blocks
      // the same within 1 %); on the training-shaped KB 3.35 -> 3.04 ms with
      // object classes (16 -> 64 blocks).
      const int32_t dr_blocks = env_int("KBFOLLOW_DR_BLOCKS", 64);
      PlanHost P[3];
      std::exception_ptr err[3];
      auto plan = [&](int k) {
        try {
          PlanOptions po;
          po.chunk = plen[k];
          po.fan_in = fan_in;
          po.n_xcd = n_xcd;
          po.hub_min = hub_min;
          po.hub_by_a = k != BY_REL;
          po.band = band;
          po.n_ids_a = n_entities;  // subjects (forward) or objects (dX, dR)
          po.class_by_b = k == BY_REL && dr_class_b;
          po.n_ids_b = n_entities;  // subjects (dR)
          po.a_blocks = k == BY_REL ? dr_blocks : 0;
          P[k] = plan_layout(H[k], po);
          H[k] = LayoutHost{H[k].rows};  // the sorted rows are no longer needed
        } catch (...) {
          err[k] = std::current_exception();
        }
      };
      {
        std::thread t1(plan, 1), t2(plan, 2);
        plan(0);
        t1.join();
        t2.join();
      }
      for (const auto &x : err)
        if (x) std::rethrow_exception(x);
      for (int k = 0; k < 3; ++k) {
        kb_status st = build_device_layout(kb, kb->L[k], H[k].rows, P[k], plen[k], s);
        if (st != KB_OK) {
          free_kb(kb);
          return st;
        }
        P[k] = PlanHost{};
      }
    }
    *out = kb;
    return KB_OK;
  } catch (const std::bad_alloc &) {
    if (kb) free_kb(kb);
    return fail(KB_ENOMEM, "host allocation failed");
  } catch (...) {
    if (kb) free_kb(kb);
    return fail(KB_EINVAL, "unexpected host error");
  }
}

void kb_destroy(kb_t *kb) {
  if (kb) free_kb(kb);
}

size_t kb_workspace_size(const kb_t *kb, int32_t b) {
  if (!kb || b < 1) return 0;
  return workspace_bytes(kb, b);
}

kb_status kb_get_info(const kb_t *kb, kb_info_t *info) {
  if (!kb || !info) return fail(KB_EINVAL, "kb and info must be non-NULL");
  std::memset(info, 0, sizeof *info);
  info->n_entities = kb->n_entities;
  info->n_relations = kb->n_relations;
  info->n_triples = kb->n_triples;
  info->weighted = kb->weighted ? 1 : 0;
  for (int k = 0; k < 3; ++k) {
    const DevLayout &D = kb->L[k];
    info->chunk_len[k] = D.chunk;
    info->n_chunks[k] = D.n_chunks;
    info->n_split_rows[k] = D.n_split_rows;
    info->n_slots[k] = D.n_slots;
    info->n_levels[k] = (int32_t)D.level_begin.size() - 1;
    info->n_empty_rows[k] = D.n_empty;
    info->max_row_len[k] = D.max_row_len;
  }
  info->device_bytes = kb->device_bytes;
  return KB_OK;
}

}  // extern "C"

namespace {

// Y = follow(X, R) [+ gamma * Z when Z is non-null].
kb_status follow_impl(const kb_t *kb, int32_t b, const float *X, const float *R, const float *Z,
                      float gamma, float *Y, void *workspace, size_t ws_bytes, void *stream) {
  try {
    if (!kb) return fail(KB_EINVAL, "kb must be non-NULL");
    if (b < 1) return fail(KB_EINVAL, "b must be >= 1");
    const size_t ent_bytes = (size_t)kb->n_entities * b * sizeof(float);
    const size_t rel_bytes = (size_t)kb->n_relations * b * sizeof(float);
    if ((ent_bytes && (!X || !Y)) || (rel_bytes && !R))
      return fail(KB_EINVAL, "X, R and Y must be non-NULL");
    const size_t al = (b % 4 == 0) ? 16 : 4;
    if ((X && !aligned(X, al)) || (R && !aligned(R, al)) || (Y && !aligned(Y, al)) ||
        (Z && !aligned(Z, al)))
      return fail(KB_EINVAL, "X, R, Z and Y must be " + std::to_string(al) + "-byte aligned");
    if (overlaps(Y, ent_bytes, X, ent_bytes) || overlaps(Y, ent_bytes, R, rel_bytes))
      return fail(KB_EINVAL, "Y overlaps X or R");
    // Row j of Z is read by the thread that then writes row j of Y: Z may be
    // Y itself, but not overlap it otherwise.
    if (Z != Y && overlaps(Z, ent_bytes, Y, ent_bytes))
      return fail(KB_EINVAL, "Z overlaps Y without being Y");
    kb_status st = check_ws(kb, b, workspace, ws_bytes,
                            {{X, ent_bytes}, {R, rel_bytes}, {Y, ent_bytes}, {Z, ent_bytes}});
    if (st != KB_OK) return st;
    if ((st = check_device(kb)) != KB_OK) return st;
    g_last_error.clear();
    if (!ent_bytes) return KB_OK;
    // By object, runs of equal relation: Y[o] = sum over runs of R[r] (.) sum of X[s].
    return run_pass(kb, kb->L[BY_OBJ], KB_PH_FWD_STREAM, X, kb->n_entities, R, kb->n_relations,
                    b, Y, workspace, Z, gamma, static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(KB_EINVAL, "unexpected host error");
  }
}

kb_status backward_impl(const kb_t *kb, int32_t b, const float *X, const float *R,
                        const float *dY, bool residual, float gamma, float *dX, float *dR,
                        void *workspace, size_t ws_bytes, void *stream) {
  try {
    if (!kb) return fail(KB_EINVAL, "kb must be non-NULL");
    if (b < 1) return fail(KB_EINVAL, "b must be >= 1");
    const size_t ent_bytes = (size_t)kb->n_entities * b * sizeof(float);
    const size_t rel_bytes = (size_t)kb->n_relations * b * sizeof(float);
    const bool want_dx = dX != nullptr && ent_bytes > 0;
    const bool want_dr = dR != nullptr && rel_bytes > 0;
    if ((want_dx || want_dr) && ent_bytes && !dY) return fail(KB_EINVAL, "dY must be non-NULL");
    if (want_dx && rel_bytes && !R) return fail(KB_EINVAL, "R must be non-NULL to compute dX");
    if (want_dr && ent_bytes && !X) return fail(KB_EINVAL, "X must be non-NULL to compute dR");
    const size_t al = (b % 4 == 0) ? 16 : 4;
    for (const void *p : {(const void *)X, (const void *)R, (const void *)dY, (const void *)dX,
                          (const void *)dR})
      if (p && !aligned(p, al))
        return fail(KB_EINVAL, "arrays must be " + std::to_string(al) + "-byte aligned");
    if (want_dx && (overlaps(dX, ent_bytes, X, ent_bytes) || overlaps(dX, ent_bytes, R, rel_bytes) ||
                    overlaps(dX, ent_bytes, dY, ent_bytes) || overlaps(dX, ent_bytes, dR, rel_bytes)))
      return fail(KB_EINVAL, "dX overlaps another array");
    if (want_dr && (overlaps(dR, rel_bytes, X, ent_bytes) || overlaps(dR, rel_bytes, R, rel_bytes) ||
                    overlaps(dR, rel_bytes, dY, ent_bytes)))
      return fail(KB_EINVAL, "dR overlaps another array");
    kb_status st = check_ws(kb, b, workspace, ws_bytes,
                            {{X, ent_bytes}, {R, rel_bytes}, {dY, ent_bytes},
                             {want_dx ? dX : nullptr, ent_bytes}, {want_dr ? dR : nullptr, rel_bytes}});
    if (st != KB_OK) return st;
    if ((st = check_device(kb)) != KB_OK) return st;
    g_last_error.clear();
    hipStream_t s = static_cast<hipStream_t>(stream);
    // dR's slots follow dX's in the workspace.  On a large KB at b <= 32
    // (or when forced) the dR pass runs on the KB's own stream, forked from
    // and joined back into the caller's: the two passes read the same dY,
    // write disjoint arrays and slots, and one's start overlaps the other's
    // tail launches.
    void *dr_ws = static_cast<char *>(workspace) + dr_slots_offset(kb, b);
    const bool overlap = want_dx && want_dr && kb->side &&
                         (kb->overlap_backward == 1 || (kb->overlap_backward == -1 && b <= 32));
    std::unique_lock<std::mutex> lock(kb->side_mu, std::defer_lock);
    hipStream_t dr_s = s;
    if (overlap) {
      lock.lock();
      hipError_t e = hipEventRecord(kb->ev_fork, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(kb->side, kb->ev_fork, 0);
      if (e != hipSuccess) return hip_fail(e, "fork of the dR pass");
      dr_s = kb->side;
    }
    if (want_dx) {
      // By subject, runs of equal relation: dX[s] = sum over runs of R[r] (.) sum of dY[o]
      // (+ gamma * dY[s] for the residual hop).
      st = run_pass(kb, kb->L[BY_SUBJ], KB_PH_DX_STREAM, dY, kb->n_entities, R, kb->n_relations,
                    b, dX, workspace, residual ? dY : nullptr, gamma, s);
    }
    if (st == KB_OK && want_dr) {
      // By relation, runs of equal subject: dR[k] = sum over runs of X[s] (.) sum of dY[o].
      st = run_pass(kb, kb->L[BY_REL], KB_PH_DR_STREAM, dY, kb->n_entities, X, kb->n_entities,
                    b, dR, dr_ws, nullptr, 0.0f, dr_s);
    }
    if (overlap) {
      // Joined whatever happened above, so the caller's stream never runs
      // ahead of work left on the KB's stream.
      hipError_t e = hipEventRecord(kb->ev_join, kb->side);
      if (e == hipSuccess) e = hipStreamWaitEvent(s, kb->ev_join, 0);
      if (e != hipSuccess && st == KB_OK) return hip_fail(e, "join of the dR pass");
    }
    return st;
  } catch (...) {
    return fail(KB_EINVAL, "unexpected host error");
  }
}

}  // namespace

extern "C" {

kb_status kb_follow(const kb_t *kb, int32_t b, const float *X, const float *R, float *Y,
                    void *workspace, size_t ws_bytes, void *stream) {
  return follow_impl(kb, b, X, R, nullptr, 0.0f, Y, workspace, ws_bytes, stream);
}

kb_status kb_follow_noalloc(const kb_t *kb, int32_t b, const float *X, const float *R, float *Y,
                            void *stream) {
  if (!kb) return fail(KB_EINVAL, "kb must be non-NULL");
  if (b < 1) return fail(KB_EINVAL, "b must be >= 1");
  // The partials go to the library's fixed scratch instead of a workspace;
  // a KB and batch size that need more than it holds are refused before
  // anything is enqueued.
  const size_t need = workspace_bytes(kb, b);
  if (need > kStaticScratchBytes)
    return fail(KB_EINVAL, "kb_follow_noalloc: this KB needs " + std::to_string(need) +
                               " bytes of scratch at b = " + std::to_string(b) +
                               ", more than the " + std::to_string(kStaticScratchBytes) +
                               " bytes of the fixed scratch (use kb_follow with a workspace)");
  kb_status st = check_device(kb);
  if (st != KB_OK) return st;
  void *ws = nullptr;
  if (need > 0) {
    hipError_t e = static_scratch(kb->device, &ws);
    if (e != hipSuccess) return hip_fail(e, "address of the fixed scratch");
  }
  return follow_impl(kb, b, X, R, nullptr, 0.0f, Y, ws, need > 0 ? kStaticScratchBytes : 0,
                     stream);
}

kb_status kb_follow_residual(const kb_t *kb, int32_t b, const float *X, const float *R,
                             float gamma, float *Y, void *workspace, size_t ws_bytes,
                             void *stream) {
  return follow_impl(kb, b, X, R, X, gamma, Y, workspace, ws_bytes, stream);
}

kb_status kb_follow_accumulate(const kb_t *kb, int32_t b, const float *X, const float *R,
                               const float *Z, float gamma, float *Y, void *workspace,
                               size_t ws_bytes, void *stream) {
  if (kb && kb->n_entities > 0 && !Z) return fail(KB_EINVAL, "Z must be non-NULL");
  return follow_impl(kb, b, X, R, Z, gamma, Y, workspace, ws_bytes, stream);
}

kb_status kb_follow_backward_residual(const kb_t *kb, int32_t b, const float *X, const float *R,
                                      const float *dY, float gamma, float *dX, float *dR,
                                      void *workspace, size_t ws_bytes, void *stream) {
  return backward_impl(kb, b, X, R, dY, true, gamma, dX, dR, workspace, ws_bytes, stream);
}

kb_status kb_follow_backward(const kb_t *kb, int32_t b, const float *X, const float *R,
                             const float *dY, float *dX, float *dR, void *workspace,
                             size_t ws_bytes, void *stream) {
  return backward_impl(kb, b, X, R, dY, false, 0.0f, dX, dR, workspace, ws_bytes, stream);
}

kb_status kb_checked_violations(uint64_t *count, int32_t reset) {
  if (!count) return fail(KB_EINVAL, "count must be non-NULL");
  *count = 0;
  unsigned long long c = 0;
  hipError_t e = checked_violations(&c, reset != 0);
  if (e == hipErrorNotSupported)
    return fail(KB_ENOTSUP, "this build has no bounds checks (build with KBFOLLOW_CHECKED)");
  if (e != hipSuccess) return hip_fail(e, "reading the violation counter");
  *count = c;
  return KB_OK;
}

kb_status kb_phase_kernel(const kb_t *kb, int32_t b, int32_t phase, int32_t residual, char *name,
                          size_t len) {
  if (!kb || !name || len == 0) return fail(KB_EINVAL, "kb and name must be non-NULL");
  if (b < 1) return fail(KB_EINVAL, "b must be >= 1");
  if (phase < 0 || phase >= KB_PH_COUNT) return fail(KB_EINVAL, "no such phase");
  try {
    kb_status st = check_device(kb);
    if (st != KB_OK) return st;
    const int pass = phase / 3, step = phase % 3;  // pass: fwd, dX, dR; step: stream, tail, combine
    const DevLayout &D = kb->L[pass == 0 ? BY_OBJ : pass == 1 ? BY_SUBJ : BY_REL];
    const bool res = residual != 0 && pass != 2;  // the dR pass has no residual term
    // Placeholder device addresses: the choice depends only on sizes, on
    // which arrays are present and on whether the added rows come from A.
    float *const A = reinterpret_cast<float *>(uintptr_t(256));
    std::string out;
    if (step == 0) {
      const int64_t B_rows = pass == 2 ? kb->n_entities : kb->n_relations;
      StreamArgs a{D.entries, D.weights, D.n,   D.chunk,    A,         kb->n_entities, A,
                   B_rows,    b,         A,     D.rows,     nullptr,   D.n_slots,      res ? 1 : 0,
                   1.0f,      res ? A : nullptr, D.n_lists, {}};
      std::copy(D.list_chunk, D.list_chunk + kMaxChunkLists + 1, a.list_chunk);
      StreamOptions o;
      o.plain_loads = kb->plain_loads;
      o.b_in_lds = kb->b_in_lds;
      o.n_cu = kb->n_cu;
      o.max_lpt = lane_cap(kb, pass * 3, b);
      out = describe_stream(a, o);
    } else if (step == 1) {
      const int64_t n0 = D.level_begin.size() > 1 ? D.level_begin[1] - D.level_begin[0] : 0;
      TailArgs t{D.ctasks, n0, nullptr, D.n_slots, D.empty, D.n_empty_pieces, b, A, D.rows,
                 res ? A : nullptr, 1.0f, 0};
      out = describe_tail(t);
    } else if (D.level_begin.size() > 2) {
      out = describe_combine(b);
    }
    std::snprintf(name, len, "%s", out.c_str());
    return KB_OK;
  } catch (...) {
    return fail(KB_EINVAL, "unexpected host error");
  }
}

kb_status kb_profile_select(kb_t *kb, uint32_t phase_mask) {
  if (!kb) return fail(KB_EINVAL, "kb must be non-NULL");
  kb_status st = kb_profile_read(kb, nullptr, nullptr);
  if (st != KB_OK) return st;
  kb->timing.mask = phase_mask & ((1u << KB_PH_COUNT) - 1u);
  return KB_OK;
}

kb_status kb_profile_enable(kb_t *kb, int32_t on) {
  return kb_profile_select(kb, on ? (1u << KB_PH_COUNT) - 1u : 0u);
}

kb_status kb_profile_read(kb_t *kb, double *ms, int64_t *launches) {
  if (!kb) return fail(KB_EINVAL, "kb must be non-NULL");
  Timing &t = kb->timing;
  kb_status st = KB_OK;
  for (auto &r : t.recs) {
    hipError_t e = hipEventSynchronize(r.stop);
    float el = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&el, r.start, r.stop);
    if (e != hipSuccess && st == KB_OK) st = hip_fail(e, "hipEventElapsedTime");
    if (ms) ms[r.phase] += el;
    if (launches) ++launches[r.phase];
    t.pool.push_back(r.start);
    t.pool.push_back(r.stop);
  }
  t.recs.clear();
  return st;
}

}  // extern "C"
