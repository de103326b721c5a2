// Host capacity policy driven by a model metric, applied at the launch
// frontier (Section 3 and its implementation appendix; Section 4.1 for the
// per-expert capacities).
//
// Every iteration the caller brackets its launches with moe_policy_begin and
// moe_policy_end.  end() enqueues a copy of the iteration's per-expert
// assignment counts (the model metric) into a pinned host ring slot and
// records an event: the metric's future.  begin() keeps exactly
// delta_launch iterations launched but not yet consumed: while more are
// outstanding it waits for the oldest future and runs the trigger on it,
// then uploads the resulting capacities and offsets (only when they changed
// or the destination buffers did) with asynchronous copies from pinned
// staging memory.  The device never waits for the host; the host waits only
// for work delta_launch iterations old, so the trigger overlaps execution.
//
// Trigger: recompile when the metric would overflow a current capacity or
// leave one above ceil(shrink * count); a recompile sets every capacity to
// ceil(grow * count), clamped to [cap_min, T].  Iteration 0 runs with the
// caller's initial capacities.
//
// Ring sizing: slots = delta_launch + 2.  The counts of iteration i sit in
// slot i mod slots until begin() of iteration i + delta_launch + 1 at the
// latest consumes them, before end() of iteration i + slots reuses the slot;
// a staging slot written at begin() of iteration i is read by a copy that
// precedes iteration i's event, which has completed before begin() of
// iteration i + slots can run.

#include <new>
#include <vector>

#include "common.hpp"
#include "validate.hpp"

struct moe_capacity_policy {
  int T = 0, k = 0, E = 0, delta = 0;
  int grow_num = 1, grow_den = 1, shrink_num = 1, shrink_den = 1, cap_min = 0;
  int row_align = 1;   // expert regions start at multiples of this many rows
  int slots = 0;
  std::vector<int32_t> cap;
  int32_t* ring = nullptr;   // pinned [slots][E] counts
  int32_t* stage = nullptr;  // pinned [slots][2E + 1] capacity, offsets
  std::vector<hipEvent_t> ev;
  int64_t launched = 0, consumed = 0, recompiles = 0;
  bool dirty = true;
  bool open = false;  // between begin() and end()
  int32_t* last_cap = nullptr;
  int32_t* last_off = nullptr;
};

namespace {

int64_t ceil_mul(int num, int den, int64_t c) { return (num * c + den - 1) / den; }

// rows an expert's region takes: its capacity rounded up to row_align
int64_t aligned_rows(int32_t cap, int row_align) {
  return (static_cast<int64_t>(cap) + row_align - 1) / row_align * row_align;
}

int32_t clamp_cap(int64_t v, int cap_min, int T) {
  if (v < cap_min) v = cap_min;
  if (v > T) v = T;
  return static_cast<int32_t>(v);
}

bool ratio_ok(int num, int den) { return num >= 1 && den >= 1 && num <= 1000000 && den <= 1000000; }

// The trigger; returns true when the capacities changed.
bool trigger(int T, int E, const int32_t* counts, int32_t* cap, int grow_num, int grow_den,
             int shrink_num, int shrink_den, int cap_min) {
  bool over = false, loose = false;
  for (int e = 0; e < E; ++e) {
    const int64_t c = counts[e];
    over = over || c > cap[e];
    loose = loose || cap[e] > clamp_cap(ceil_mul(shrink_num, shrink_den, c), cap_min, T);
  }
  if (!over && !loose) return false;
  for (int e = 0; e < E; ++e)
    cap[e] = clamp_cap(ceil_mul(grow_num, grow_den, counts[e]), cap_min, T);
  return true;
}

void release(moe_capacity_policy* p) {
  for (hipEvent_t e : p->ev)
    if (e) (void)hipEventDestroy(e);
  if (p->ring) (void)hipHostFree(p->ring);
  if (p->stage) (void)hipHostFree(p->stage);
  delete p;
}

}  // namespace

extern "C" int moe_capacity_trigger(int T, int E, const int32_t* counts, int32_t* cap,
                                    int grow_num, int grow_den, int shrink_num, int shrink_den,
                                    int cap_min) {
  if (T < 0 || E < 1 || E > moe::kMaxE || !counts || !cap || cap_min < 0) return -1;
  if (!ratio_ok(grow_num, grow_den) || !ratio_ok(shrink_num, shrink_den)) return -1;
  if (static_cast<int64_t>(grow_num) * shrink_den > static_cast<int64_t>(shrink_num) * grow_den)
    return -1;
  for (int e = 0; e < E; ++e)
    if (counts[e] < 0 || cap[e] < 0) return -1;
  return trigger(T, E, counts, cap, grow_num, grow_den, shrink_num, shrink_den, cap_min) ? 1 : 0;
}

extern "C" moe_status moe_policy_create(int T, int k, int E, int delta_launch, int grow_num,
                                        int grow_den, int shrink_num, int shrink_den,
                                        int cap_min, int row_align, const int32_t* init_cap,
                                        moe_capacity_policy** out) {
  using namespace moe;
  if (!out) return MOE_EINVAL;
  *out = nullptr;
  if (!shape_ok(T, E, k) || delta_launch < 0 || delta_launch > 64 || !init_cap) return MOE_EINVAL;
  if (!ratio_ok(grow_num, grow_den) || !ratio_ok(shrink_num, shrink_den) || cap_min < 0)
    return MOE_EINVAL;
  if (row_align < 1 || row_align > kMaxRowAlign) return MOE_EINVAL;
  // grow <= shrink: a recompile never leaves a capacity the same metric would shrink
  if (static_cast<int64_t>(grow_num) * shrink_den > static_cast<int64_t>(shrink_num) * grow_den)
    return MOE_EINVAL;
  moe_capacity_policy* p = new (std::nothrow) moe_capacity_policy;
  if (!p) return MOE_EHIP;
  p->T = T; p->k = k; p->E = E; p->delta = delta_launch;
  p->grow_num = grow_num; p->grow_den = grow_den;
  p->shrink_num = shrink_num; p->shrink_den = shrink_den; p->cap_min = cap_min;
  p->row_align = row_align;
  p->slots = delta_launch + 2;
  p->cap.resize(E);
  for (int e = 0; e < E; ++e) {
    if (init_cap[e] < 0) { release(p); return MOE_EINVAL; }
    p->cap[e] = clamp_cap(init_cap[e], cap_min, T);
  }
  if (hipHostMalloc(reinterpret_cast<void**>(&p->ring),
                    sizeof(int32_t) * p->slots * E) != hipSuccess ||
      hipHostMalloc(reinterpret_cast<void**>(&p->stage),
                    sizeof(int32_t) * p->slots * (2 * E + 1)) != hipSuccess) {
    release(p);
    return MOE_EHIP;
  }
  p->ev.assign(p->slots, nullptr);
  for (int i = 0; i < p->slots; ++i)
    if (hipEventCreateWithFlags(&p->ev[i], hipEventDisableTiming) != hipSuccess) {
      release(p);
      return MOE_EHIP;
    }
  *out = p;
  return MOE_OK;
}

extern "C" void moe_policy_destroy(moe_capacity_policy* p) {
  if (!p) return;
  // the copies still in flight write into the ring: wait for them
  for (int64_t i = p->consumed; i < p->launched; ++i)
    (void)hipEventSynchronize(p->ev[i % p->slots]);
  release(p);
}

extern "C" moe_status moe_policy_begin(moe_capacity_policy* p, void* stream, int32_t* capacity,
                                       int32_t* offsets, int64_t* rows_needed,
                                       int* recompiled) {
  if (!p || !capacity || !offsets || p->open) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  bool changed = false;
  while (p->launched - p->consumed > p->delta) {
    const int slot = static_cast<int>(p->consumed % p->slots);
    if (hipEventSynchronize(p->ev[slot]) != hipSuccess) return MOE_EHIP;
    if (trigger(p->T, p->E, p->ring + static_cast<size_t>(slot) * p->E, p->cap.data(),
                p->grow_num, p->grow_den, p->shrink_num, p->shrink_den, p->cap_min)) {
      changed = true;
      ++p->recompiles;
    }
    ++p->consumed;
  }
  if (changed || p->dirty || capacity != p->last_cap || offsets != p->last_off) {
    const int slot = static_cast<int>(p->launched % p->slots);
    int32_t* st = p->stage + static_cast<size_t>(slot) * (2 * p->E + 1);
    int64_t acc = 0;
    for (int e = 0; e < p->E; ++e) {
      st[e] = p->cap[e];
      st[p->E + e] = static_cast<int32_t>(acc);
      acc += aligned_rows(p->cap[e], p->row_align);
    }
    if (acc >= (int64_t(1) << 31)) {
      p->dirty = true;  // the capacities were not uploaded
      return MOE_EINVAL;
    }
    st[2 * p->E] = static_cast<int32_t>(acc);
    if (hipMemcpyAsync(capacity, st, sizeof(int32_t) * p->E, hipMemcpyHostToDevice, s) !=
            hipSuccess ||
        hipMemcpyAsync(offsets, st + p->E, sizeof(int32_t) * (p->E + 1), hipMemcpyHostToDevice,
                       s) != hipSuccess)
      return MOE_EHIP;
    p->dirty = false;
    p->last_cap = capacity;
    p->last_off = offsets;
  }
  if (rows_needed) {
    int64_t acc = 0;
    for (int e = 0; e < p->E; ++e) acc += aligned_rows(p->cap[e], p->row_align);
    *rows_needed = acc;
  }
  if (recompiled) *recompiled = changed ? 1 : 0;
  p->open = true;
  return MOE_OK;
}

extern "C" moe_status moe_policy_end(moe_capacity_policy* p, void* stream,
                                     const int32_t* counts) {
  if (!p || !counts || !p->open) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int slot = static_cast<int>(p->launched % p->slots);
  if (hipMemcpyAsync(p->ring + static_cast<size_t>(slot) * p->E, counts,
                     sizeof(int32_t) * p->E, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipEventRecord(p->ev[slot], s) != hipSuccess)
    return MOE_EHIP;
  ++p->launched;
  p->open = false;
  return MOE_OK;
}

extern "C" moe_status moe_policy_state(const moe_capacity_policy* p, int32_t* cap,
                                       int64_t* launched, int64_t* consumed,
                                       int64_t* recompiles) {
  if (!p) return MOE_EINVAL;
  if (cap)
    for (int e = 0; e < p->E; ++e) cap[e] = p->cap[e];
  if (launched) *launched = p->launched;
  if (consumed) *consumed = p->consumed;
  if (recompiles) *recompiles = p->recompiles;
  return MOE_OK;
}
