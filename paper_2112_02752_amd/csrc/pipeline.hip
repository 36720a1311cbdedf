// The pipelined training schedule, enqueued natively: the id dedups of each
// next group of batches on side streams while the main stream runs the
// forward and the fused update of the current group.  The dedup reads only a
// batch's ids and offsets, never the table, so running it early changes no
// result.  Everything here is host code that only enqueues work through the
// library's entry points and HIP events (no allocation, no synchronisation
// with the device).
//
// Enqueueing a dedup costs the host tens of microseconds (a dozen kernel
// launches for the wait-free dedup), about as long as the device takes for a
// whole step, so with more than one group each side stream's work is
// enqueued by a helper thread of its own while the calling thread enqueues
// the main stream's (kernel launches on different streams proceed in
// parallel from different threads).  Counters keep every cross-stream wait
// attached to the same event record as in a single-threaded enqueue:
//   side_done[s]: groups whose dedups and record on side stream s are
//     enqueued; the main stream's waits for group g are enqueued only once
//     every side_done[s] > g.
//   main_done: groups whose main-stream record is enqueued; the dedups of
//     group g >= P (which reuse the buffer sets of group g - P; P = depth,
//     the number of buffer set parities) are enqueued only once
//     main_done >= g - P + 1, after their wait for that record.
// The side thread re-records the events of a parity only after the main
// thread has enqueued its wait on the previous record (main_done >= g - P + 1
// implies the main stream's wait for group g - P is enqueued), so no wait
// ever attaches to a later record, which could make the two streams wait
// for each other.
//
// Calls can be chained (a training loop's look-ahead): a call may end with
// the dedups of the A < P groups of batches after its steps (ahead), into
// the buffer sets the next call's first groups read, and the next call then
// starts with those dedups already enqueued (primed).  Groups are numbered
// across calls (group_base) so that buffer parities rotate across the
// boundary; the look-ahead dedups wait like any others for the main stream's
// group of the same parity, and the next call's first groups wait for them
// through the same events.  Every side stream of a call still starts after
// the work already on the main stream, so the batches it reads may be
// written there until the call that dedups them.
#include <atomic>
#include <system_error>
#include <thread>

#include "emb_common.h"
#include "kernels.h"

namespace {

constexpr int kMaxSideStreams = 16;  // one host thread each
constexpr int kMaxDepth = 8;         // buffer set parities

struct Schedule {
  const emb_tables* tables;
  int32_t pool;
  const emb_update* update;
  int32_t n_steps, K, ngroups, n_side;
  const emb_batch* batches;
  float* const* outs;
  const float* const* grads;
  const emb_dedup_set* sets;
  hipStream_t main;
  void* const* sides;
  hipEvent_t ev_start;
  void* const* events;  // [1 + depth + depth * n_side]: start, main per parity, side per parity and stream
  void* group_ws;  // non-null: each group's dedups as one emb_unique_ids_batched call
  size_t group_ws_bytes;
  int32_t depth;       // buffer set parities (groups whose sets are in use at once)
  int32_t group_base;  // this call's first group in the numbering across calls (buffer parity)
  int32_t primed;      // the first groups whose dedups were enqueued by the previous call
  int32_t ahead;       // groups of K batches after the steps (batches[n_steps...]) also deduped

  hipEvent_t ev_main(int parity) const { return (hipEvent_t)events[1 + parity]; }
  hipEvent_t ev_side(int parity, int s) const { return (hipEvent_t)events[1 + depth + parity * n_side + s]; }
  hipStream_t side(int s) const { return (hipStream_t)sides[s]; }
  int parity(int g) const { return (group_base + g) % depth; }
  // group g < ngroups: steps [g K, min(g K + K, n_steps)); group ngroups + j
  // (j < ahead): the j-th K look-ahead batches
  int start(int g) const { return g < ngroups ? g * K : n_steps + (g - ngroups) * K; }
  int count(int g) const { return g < ngroups ? (n_steps - g * K < K ? n_steps - g * K : K) : K; }
  int side_first() const { return primed; }
  int side_end() const { return ngroups + ahead; }
};

emb_status hip_ok(hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_EHIP; }

// one dedup in flight per side stream at most with emb_unique_ids (which may
// make the workgroups of a pass wait for one another); several side streams
// use emb_unique_ids_concurrent, whose workgroups never wait for one another
emb_status dedup_one(const Schedule& c, int k, const emb_dedup_set& d, void* stream) {
  auto fn = c.n_side > 1 ? emb_unique_ids_concurrent : emb_unique_ids;
  return fn(c.tables, &c.batches[k], d.unique_keys, d.counts, d.seg_offsets, d.sort_perm, d.num_unique, d.ws,
            d.ws_bytes, stream);
}

// side stream s's part of group g: (for g >= depth) its wait for the main
// stream's group g - depth, the dedups of the group dealt to it
// (i % n_side == s) into the buffer sets of the group's parity, and its
// record (groups below depth follow the call's start, and so every earlier
// group of the main stream)
emb_status side_group(const Schedule& c, int g, int s) {
  const int par = c.parity(g);
  if (g >= c.depth && hipStreamWaitEvent(c.side(s), c.ev_main(par), 0) != hipSuccess) return EMB_EHIP;
  if (c.group_ws != nullptr) {
    // a group of one batch: its own dedup (one dedup in flight on this
    // stream, beside kernels that never wait)
    const emb_status r = c.count(g) == 1
                             ? emb_unique_ids(c.tables, &c.batches[c.start(g)], c.sets[par * c.K].unique_keys,
                                              c.sets[par * c.K].counts, c.sets[par * c.K].seg_offsets,
                                              c.sets[par * c.K].sort_perm, c.sets[par * c.K].num_unique,
                                              c.sets[par * c.K].ws, c.sets[par * c.K].ws_bytes, c.sides[s])
                             : emb_unique_ids_batched(c.tables, c.count(g), &c.batches[c.start(g)], &c.sets[par * c.K],
                                                      c.group_ws, c.group_ws_bytes, c.sides[s]);
    if (r != EMB_OK) return r;
    return hip_ok(hipEventRecord(c.ev_side(par, s), c.side(s)));
  }
  for (int i = s; i < c.count(g); i += c.n_side) {
    const emb_status r = dedup_one(c, c.start(g) + i, c.sets[par * c.K + i], c.sides[s]);
    if (r != EMB_OK) return r;
  }
  return hip_ok(hipEventRecord(c.ev_side(par, s), c.side(s)));
}

emb_status side_group_all(const Schedule& c, int g) {
  for (int s = 0; s < c.n_side; ++s) {
    const emb_status r = side_group(c, g, s);
    if (r != EMB_OK) return r;
  }
  return EMB_OK;
}

// The main stream's part of group g: each step's forward and fused backward
// + update, then the group's record.  The group's first forward reads no
// dedup output, so it comes before the wait for the group's dedups (and, in
// the threaded enqueue, before the host waits for their record).
emb_status main_first_forward(const Schedule& c, int g) {
  const int k = c.start(g);
  return emb_pool_fwd(c.tables, &c.batches[k], c.pool, c.outs[k], c.main);
}

emb_status main_group_rest(const Schedule& c, int g) {
  const int par = c.parity(g);
  for (int s = 0; s < c.n_side; ++s)
    if (hipStreamWaitEvent(c.main, c.ev_side(par, s), 0) != hipSuccess) return EMB_EHIP;
  emb_update u = *c.update;
  for (int i = 0; i < c.count(g); ++i) {
    const int k = c.start(g) + i;
    const emb_dedup_set& d = c.sets[par * c.K + i];
    u.seed = c.update->seed + (uint64_t)k;  // bf16 stochastic rounding draws fresh bits every step
    emb_status st = i > 0 ? emb_pool_fwd(c.tables, &c.batches[k], c.pool, c.outs[k], c.main) : EMB_OK;
    if (st == EMB_OK)
      st = emb_grad_reduce(c.tables, &c.batches[k], c.pool, c.grads[k], d.sort_perm, d.seg_offsets, d.unique_keys,
                           d.num_unique, nullptr, &u, d.ws, d.ws_bytes, c.main);
    if (st != EMB_OK) return st;
  }
  return hip_ok(hipEventRecord(c.ev_main(par), c.main));
}

emb_status main_group(const Schedule& c, int g) {
  const emb_status st = main_first_forward(c, g);
  return st == EMB_OK ? main_group_rest(c, g) : st;
}

// the main stream's last waits of a call with look-ahead dedups: for them, so
// that the end of the main stream's work is the end of all the call's work
emb_status main_join_ahead(const Schedule& c) {
  for (int j = 0; j < c.ahead; ++j)
    for (int s = 0; s < c.n_side; ++s)
      if (hipStreamWaitEvent(c.main, c.ev_side(c.parity(c.ngroups + j), s), 0) != hipSuccess) return EMB_EHIP;
  return EMB_OK;
}

// single thread, from the main stream's group g_first on, with the side
// streams' part of every group below next_side enqueued (or primed): the side
// part of each group up to g + 1 before the main stream's part of group g,
// then the side part of the remaining look-ahead groups
emb_status run_single_from(const Schedule& c, int g_first, int next_side) {
  emb_status st = EMB_OK;
  for (int g = g_first; g < c.ngroups && st == EMB_OK; ++g) {
    for (; next_side <= g + 1 && next_side < c.side_end() && st == EMB_OK; ++next_side)
      st = side_group_all(c, next_side);
    if (st == EMB_OK) st = main_group(c, g);
  }
  for (; next_side < c.side_end() && st == EMB_OK; ++next_side) st = side_group_all(c, next_side);
  return st == EMB_OK ? main_join_ahead(c) : st;
}

// side stream s's wait for the call's start record, enqueued just before its
// first work by the thread that enqueues that work (the wait costs the host
// 15-25 us, which stays off the main stream's first launches)
emb_status side_wait_start(const Schedule& c, int s) {
  return hip_ok(hipStreamWaitEvent(c.side(s), c.ev_start, 0));
}

emb_status run_single(const Schedule& c) {
  for (int s = 0; s < c.n_side; ++s)
    if (side_wait_start(c, s) != EMB_OK) return EMB_EHIP;
  const emb_status st = c.side_first() == 0 ? side_group_all(c, 0) : EMB_OK;
  return st == EMB_OK ? run_single_from(c, 0, c.side_first() > 1 ? c.side_first() : 1) : st;
}

bool await_count(const std::atomic<int>& n, int v, const std::atomic<int>& failed) {
  while (n.load(std::memory_order_acquire) < v) {
    if (failed.load(std::memory_order_acquire)) return false;
    std::this_thread::yield();
  }
  return true;
}

emb_status run_threaded(const Schedule& c) {
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess) return EMB_EHIP;
  std::atomic<int> side_done[kMaxSideStreams], main_done{0}, failed{0};
  emb_status side_st[kMaxSideStreams];
  for (int s = 0; s < c.n_side; ++s) {
    side_done[s].store(c.side_first());
    side_st[s] = EMB_OK;
  }
  auto side_work = [&](int s) {
    // the current device is per thread: the caller's
    if (hipSetDevice(device) != hipSuccess || side_wait_start(c, s) != EMB_OK) {
      side_st[s] = EMB_EHIP;
      failed.store(1, std::memory_order_release);
      return;
    }
    for (int g = c.side_first(); g < c.side_end(); ++g) {
      if (failed.load(std::memory_order_acquire)) return;
      if (g >= c.depth && !await_count(main_done, g - c.depth + 1, failed)) return;
      side_st[s] = side_group(c, g, s);
      if (side_st[s] != EMB_OK) {
        failed.store(1, std::memory_order_release);
        return;
      }
      side_done[s].store(g + 1, std::memory_order_release);
    }
  };
  // With the first group's dedups enqueued by the previous call, its main
  // stream work goes first, before any helper thread starts: the device then
  // has work at once instead of after the helpers' first launches (launches
  // from several threads take turns).  The helpers' first group (primed)
  // waits for nothing of the main stream's (primed < depth).
  emb_status st = EMB_OK;
  int g_first = 0;
  if (c.primed) {
    if ((st = main_group(c, 0)) != EMB_OK) return st;
    main_done.store(1, std::memory_order_release);
    g_first = 1;
  }
  std::thread helpers[kMaxSideStreams];
  int started = 0;
  try {
    for (; started < c.n_side; ++started) helpers[started] = std::thread(side_work, started);
  } catch (const std::system_error&) {
    failed.store(1, std::memory_order_release);
    for (int s = 0; s < started; ++s) helpers[s].join();
    // with no thread started, no dedup of this call is enqueued yet: the rest
    // of the schedule from this thread (a primed call's first group is
    // already enqueued); otherwise the started ones may have enqueued dedups
    // of the next groups (which nothing waits on) and the call fails
    if (started > 0) return EMB_EHIP;
    if (g_first == 0) return run_single(c);
    for (int s = 0; s < c.n_side; ++s)
      if (side_wait_start(c, s) != EMB_OK) return EMB_EHIP;
    // the primed first group's main stream work is enqueued: the rest in
    // the single-thread order, the side streams' from the first group not
    // primed
    return run_single_from(c, 1, c.side_first());
  }
  for (int g = g_first; g < c.ngroups && st == EMB_OK; ++g) {
    if ((st = main_first_forward(c, g)) != EMB_OK) {
      failed.store(1, std::memory_order_release);
      break;
    }
    for (int s = 0; s < c.n_side; ++s)
      if (!await_count(side_done[s], g + 1, failed)) st = EMB_EHIP;
    if (st != EMB_OK) break;
    if ((st = main_group_rest(c, g)) != EMB_OK) {
      failed.store(1, std::memory_order_release);
      break;
    }
    main_done.store(g + 1, std::memory_order_release);
  }
  if (st == EMB_OK && c.ahead) {
    for (int s = 0; s < c.n_side; ++s)
      if (!await_count(side_done[s], c.side_end(), failed)) st = EMB_EHIP;
    if (st == EMB_OK) st = main_join_ahead(c);
  }
  for (int s = 0; s < c.n_side; ++s) helpers[s].join();
  for (int s = 0; s < c.n_side; ++s)
    if (side_st[s] != EMB_OK) return side_st[s];
  return st;
}

}  // namespace

extern "C" {

emb_status emb_pipeline_steps(const emb_tables* tables, int32_t pool, const emb_update* update, int32_t n_steps,
                              const emb_batch* batches, float* const* outs, const float* const* grads,
                              int32_t group, const emb_dedup_set* sets, void* main_stream, int32_t n_side,
                              void* const* side_streams, void* const* events, void* group_ws,
                              size_t group_ws_bytes, int32_t group_base, int32_t primed, int32_t ahead,
                              int32_t depth) {
  if (tables == nullptr || update == nullptr || n_steps < 0 || group < 1 || n_side < 1 || n_side > group ||
      depth < 2 || group_base < 0 || primed < 0 || primed >= depth || ahead < 0 || ahead >= depth)
    return EMB_EINVAL;
  if (n_side > kMaxSideStreams || depth > kMaxDepth) return EMB_EUNSUPPORTED;
  if (group_ws != nullptr && n_side != 1) return EMB_EINVAL;  // a group's one dedup runs on one stream
  if (group_ws != nullptr && group > emb::kMaxGroup) return EMB_EUNSUPPORTED;
  if (n_steps == 0) return ahead ? EMB_EINVAL : EMB_OK;
  // the primed groups are whole groups of this call's first steps
  if ((int64_t)primed * group > n_steps) return EMB_EINVAL;
  if (batches == nullptr || outs == nullptr || grads == nullptr || sets == nullptr || side_streams == nullptr ||
      events == nullptr)
    return EMB_EINVAL;
  for (int i = 0; i < 1 + depth + depth * n_side; ++i)
    if (events[i] == nullptr) return EMB_EINVAL;
  for (int s = 0; s < n_side; ++s)
    if (side_streams[s] == nullptr || side_streams[s] == main_stream) return EMB_EINVAL;
  Schedule c{};
  c.tables = tables;
  c.pool = pool;
  c.update = update;
  c.n_steps = n_steps;
  c.K = group;
  c.ngroups = (n_steps + group - 1) / group;
  c.n_side = n_side;
  c.batches = batches;
  c.outs = outs;
  c.grads = grads;
  c.sets = sets;
  c.main = (hipStream_t)main_stream;
  c.sides = side_streams;
  c.ev_start = (hipEvent_t)events[0];
  c.events = events;
  c.depth = depth;
  c.group_ws = group_ws;
  c.group_ws_bytes = group_ws_bytes;
  c.group_base = group_base;
  c.primed = primed;
  c.ahead = ahead;
  // every step, and every look-ahead batch's dedup, is checked before
  // anything is enqueued
  for (int g = 0; g < c.side_end(); ++g) {
    for (int i = 0; i < c.count(g); ++i) {
      const int k = c.start(g) + i;
      const emb_dedup_set* d = &sets[c.parity(g) * group + i];
      const emb_status st = g < c.ngroups
                                ? emb::check_pipeline_step(tables, &batches[k], pool, outs[k], grads[k], update, d)
                                : emb::check_dedup_step(tables, &batches[k], d);
      if (st != EMB_OK) return st;
    }
    if (group_ws != nullptr && g >= c.side_first()) {
      const emb_status st = emb::check_dedup_group(tables, c.count(g), &batches[c.start(g)], group_ws, group_ws_bytes);
      if (st != EMB_OK) return st;
    }
  }
  // the side streams start after the work already on the main stream (their
  // waits for this record are enqueued by whichever thread enqueues their work)
  if (hipEventRecord(c.ev_start, c.main) != hipSuccess) return EMB_EHIP;
  return c.ngroups + c.ahead > 1 ? run_threaded(c) : run_single(c);
}

}  // extern "C"
