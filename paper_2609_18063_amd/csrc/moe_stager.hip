// Host-tier expert staging (include/moe_api.h, "host-tier staging").
//
// The paper's staged executor keeps a fixed set of slots per layer and
// rewrites only the slots whose expert changed (Sec. 3.1, Executor paths);
// the prerouter's prediction for layer N+1 at token t+1 lets that rewrite
// start one token early (Sec. 3.2, Motivation).  Here the experts of the
// 8B tier live in pinned host memory, a layer has a small pool of device
// slots, and:
//
//   moe_slot_policy   which slot each needed expert goes to (host logic).
//   moe_stager        the policy plus the work it implies on the GPU: the
//                     layer's slot-table rows are rewritten on the device and
//                     each missing bundle is copied host -> slot with
//                     hipMemcpyAsync on a copy stream; an event per staged
//                     set lets the compute stream wait for exactly its copies.
//
// File tier (Sec. 3.1, SSD streaming; the paper maps per-layer stacked
// weight files and reads experts through the OS page cache): with
// moe_stager_create_file the bundles live in one file, [L][n_ids] records of
// file_stride bytes, mapped read-only. A copy reads the record from the
// mapping into one of a ring of pinned bounce buffers (page faults read the
// file, or hit the page cache), split over a few host threads, then
// hipMemcpyAsync moves it to the slot; a bounce buffer is reused only after
// the event recorded behind its copy. The reads run on the stager's I/O
// thread, in the order the sets were staged, so that staging does not hold up
// the thread that launches the kernels.
//
// Policy (the paper leaves it open; the reading is stated once here and in
// the header): every layer keeps a FIFO of staged-but-unused sets and a FIFO
// of sets in use.  Staging a set walks it in routing order; a resident expert
// costs nothing; a missing one takes the lowest free slot, else the slot with
// the oldest last use among the unpinned slots (ties to the lowest slot id).
// Pinned: the slots of the set being staged, of every set still queued and of
// every set in use (used, and not yet released: its kernels may still read
// it).  A clock that advances on every copy and every use orders "last use".
#include <hip/hip_runtime.h>

#include <fcntl.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "moe_table.h"

struct moe_slot_policy {
  int n_layers = 0, n_ids = 0, n_slots = 0;
  std::vector<int32_t> slot_of;     // [L][n_ids], -1 = not resident
  std::vector<int32_t> expert_in;   // [L][n_slots], -1 = free
  std::vector<int64_t> last_use;    // [L][n_slots]
  std::vector<std::deque<std::vector<int32_t>>> pending;  // [L] FIFO of staged sets
  std::vector<std::deque<std::vector<int32_t>>> in_use;   // [L] FIFO of sets in use
  int64_t clock = 0;
};

namespace {

bool set_ok(const moe_slot_policy* p, int layer, const int32_t* e, int n) {
  if (!p || layer < 0 || layer >= p->n_layers || n < 0 || (n > 0 && !e)) return false;
  for (int i = 0; i < n; ++i) {
    if (e[i] < 0 || e[i] >= p->n_ids) return false;
    for (int j = 0; j < i; ++j)
      if (e[j] == e[i]) return false;  // a routing set has distinct experts
  }
  return true;
}

// Stage: returns the number of copies written to `copies` as (expert, slot)
// pairs, or a negative error (then nothing changed).
int policy_stage(moe_slot_policy* p, int layer, const int32_t* e, int n, int32_t* copies) {
  if (!set_ok(p, layer, e, n)) return MOE_EINVAL;
  int32_t* so = &p->slot_of[(size_t)layer * p->n_ids];
  int32_t* ei = &p->expert_in[(size_t)layer * p->n_slots];
  int64_t* lu = &p->last_use[(size_t)layer * p->n_slots];
  std::vector<char> pinned(p->n_slots, 0);
  auto pin_set = [&](const int32_t* s, int m) {
    for (int i = 0; i < m; ++i)
      if (so[s[i]] >= 0) pinned[so[s[i]]] = 1;
  };
  pin_set(e, n);
  for (const auto& q : p->pending[layer]) pin_set(q.data(), (int)q.size());
  for (const auto& q : p->in_use[layer]) pin_set(q.data(), (int)q.size());
  // check capacity first so that a failing call changes nothing
  int missing = 0, free_slots = 0, evictable = 0;
  for (int i = 0; i < n; ++i) missing += so[e[i]] < 0;
  for (int s = 0; s < p->n_slots; ++s) {
    free_slots += ei[s] < 0;
    evictable += ei[s] >= 0 && !pinned[s];
  }
  if (missing > free_slots + evictable) return MOE_ENOMEM;
  int nc = 0;
  for (int i = 0; i < n; ++i) {
    const int x = e[i];
    if (so[x] >= 0) continue;
    int slot = -1;
    for (int s = 0; s < p->n_slots && slot < 0; ++s)
      if (ei[s] < 0) slot = s;
    if (slot < 0) {
      for (int s = 0; s < p->n_slots; ++s)
        if (!pinned[s] && (slot < 0 || lu[s] < lu[slot])) slot = s;
      so[ei[slot]] = -1;  // evicted
    }
    so[x] = slot;
    ei[slot] = x;
    pinned[slot] = 1;
    lu[slot] = ++p->clock;
    if (copies) {
      copies[2 * nc] = x;
      copies[2 * nc + 1] = slot;
    }
    ++nc;
  }
  p->pending[layer].emplace_back(e, e + n);
  return nc;
}

int policy_use(moe_slot_policy* p, int layer, const int32_t* e, int n, int32_t* slots) {
  if (!set_ok(p, layer, e, n)) return MOE_EINVAL;
  auto& q = p->pending[layer];
  if (q.empty() || (int)q.front().size() != n || !std::equal(q.front().begin(), q.front().end(), e))
    return MOE_EINVAL;  // not the oldest staged set of the layer
  const int32_t* so = &p->slot_of[(size_t)layer * p->n_ids];
  for (int i = 0; i < n; ++i)
    if (so[e[i]] < 0) return MOE_ENOTRESIDENT;
  p->in_use[layer].push_back(std::move(q.front()));
  q.pop_front();
  int64_t* lu = &p->last_use[(size_t)layer * p->n_slots];
  for (int i = 0; i < n; ++i) {
    lu[so[e[i]]] = ++p->clock;
    if (slots) slots[i] = so[e[i]];
  }
  return MOE_OK;
}

int policy_release(moe_slot_policy* p, int layer) {
  if (!p || layer < 0 || layer >= p->n_layers || p->in_use[layer].empty()) return MOE_EINVAL;
  p->in_use[layer].pop_front();
  return MOE_OK;
}

}  // namespace

int moe_slot_policy_create(int n_layers, int n_ids, int n_slots, moe_slot_policy** out) {
  if (!out || n_layers < 1 || n_ids < 1 || n_slots < 1) return MOE_EINVAL;
  moe_slot_policy* p = new (std::nothrow) moe_slot_policy;
  if (!p) return MOE_ENOMEM;
  p->n_layers = n_layers;
  p->n_ids = n_ids;
  p->n_slots = n_slots;
  p->slot_of.assign((size_t)n_layers * n_ids, -1);
  p->expert_in.assign((size_t)n_layers * n_slots, -1);
  p->last_use.assign((size_t)n_layers * n_slots, -1);
  p->pending.resize(n_layers);
  p->in_use.resize(n_layers);
  *out = p;
  return MOE_OK;
}

int moe_slot_policy_destroy(moe_slot_policy* p) {
  delete p;
  return MOE_OK;
}

int moe_slot_policy_stage(moe_slot_policy* p, int layer, const int32_t* experts, int n,
                          int32_t* copies) {
  return policy_stage(p, layer, experts, n, copies);
}

int moe_slot_policy_use(moe_slot_policy* p, int layer, const int32_t* experts, int n,
                        int32_t* slots) {
  return policy_use(p, layer, experts, n, slots);
}

int moe_slot_policy_release(moe_slot_policy* p, int layer) { return policy_release(p, layer); }

int moe_slot_policy_lookup(const moe_slot_policy* p, int layer, int expert) {
  if (!p || layer < 0 || layer >= p->n_layers || expert < 0 || expert >= p->n_ids)
    return MOE_EINVAL;
  const int s = p->slot_of[(size_t)layer * p->n_ids + expert];
  return s >= 0 ? s : MOE_ENOTRESIDENT;
}

// ---------------------------------------------------------------------------
struct moe_stager {
  moe_slot_table* table = nullptr;
  moe_slot_policy* policy = nullptr;
  moe_bundle_layout layout{};
  size_t bundle_bytes = 0, slot_stride = 0;
  std::vector<const void*> host;   // [L][n_ids]
  char* pool = nullptr;            // device [L][n_slots][slot_stride]
  // pinned staging ring for the table rows written to the device
  size_t row_bytes = 0, row_so_bytes = 0;
  char* ring = nullptr;
  std::vector<hipEvent_t> ring_ev;
  std::vector<char> ring_used;
  int ring_next = 0;
  // one event per staged set, FIFO per layer (parallel to the policy's
  // queue); null when the set needed no copy.  Retired events are reused
  // only after kRetire later retirements.
  std::vector<std::deque<hipEvent_t>> set_ev;
  std::deque<hipEvent_t> free_ev;
  moe_stager_stats stats{};
  // file tier (map == nullptr: pinned host bundles)
  int fd = -1;
  const char* map = nullptr;
  size_t map_bytes = 0, file_stride = 0, bounce_stride = 0;
  char* bounce = nullptr;
  int n_bounce = 0, bounce_next = 0, n_io = 1;
  std::vector<hipEvent_t> bounce_ev;
  std::vector<char> bounce_used;
  std::atomic<int64_t> read_ns{0}, read_bytes{0};
  // File tier: one I/O thread takes the staged sets in order, reads their
  // records and issues their copies, so that stage() returns at once and the
  // launching thread keeps launching. use() waits (on the host) only until
  // the set's copies are issued, then makes the compute stream wait for them.
  struct IoJob {
    int layer = 0;
    std::vector<int32_t> cp;  // (expert, slot) pairs
    hipEvent_t ev = nullptr;  // recorded after the set's copies
    hipStream_t st = nullptr;
    uint64_t seq = 0;
  };
  std::thread io;
  std::mutex mu;
  std::condition_variable cv_job, cv_issued;
  std::deque<IoJob> jobs;
  uint64_t next_seq = 0, issued = 0;           // sets with seq < issued are issued
  bool stop = false;
  std::vector<std::deque<uint64_t>> set_seq;  // [L] FIFO parallel to set_ev (file tier)
  int device = 0;
  // A copy could not be issued after the table and the policy had taken the
  // set: the slots no longer hold what the table says, so every later stage
  // and use fails with MOE_EHIP.
  std::atomic<bool> failed{false};
};

namespace {

constexpr int kRing = 64;
constexpr size_t kRetire = 32;
constexpr uint64_t kNoJob = ~(uint64_t)0;  // a set that needed no copy

hipEvent_t take_event(moe_stager* s) {
  if (s->free_ev.size() > kRetire) {
    hipEvent_t e = s->free_ev.front();
    s->free_ev.pop_front();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
  return e;
}

bool layout_ok(const moe_bundle_layout* l, size_t bytes) {
  const int64_t* f[3] = {l->gate, l->up, l->down};
  for (const int64_t* p : f) {
    for (int i = 0; i < 4; ++i) {
      if (i < 2 && p[i] < 0) return false;  // codes and scales are required
      if (p[i] >= 0 && ((p[i] & 15) != 0 || (size_t)p[i] >= bytes)) return false;
    }
    if ((p[2] < 0) != (p[3] < 0)) return false;  // LoRA needs both factors
  }
  return true;
}

moe_bundle slot_bundle(const moe_stager* s, int layer, int slot) {
  const char* base = s->pool + ((size_t)layer * s->table->n_slots + slot) * s->slot_stride;
  auto at = [&](int64_t off) -> const void* { return off < 0 ? nullptr : base + off; };
  const moe_bundle_layout& l = s->layout;
  moe_bundle b;
  b.gate = moe_proj{at(l.gate[0]), at(l.gate[1]), at(l.gate[2]), at(l.gate[3])};
  b.up = moe_proj{at(l.up[0]), at(l.up[1]), at(l.up[2]), at(l.up[3])};
  b.down = moe_proj{at(l.down[0]), at(l.down[1]), at(l.down[2]), at(l.down[3])};
  return b;
}

// Writes the layer's rows of the slot table (host mirror -> pinned ring ->
// device) on `st`.
int push_rows(moe_stager* s, int layer, hipStream_t st) {
  moe_slot_table* t = s->table;
  const int r = s->ring_next;
  s->ring_next = (r + 1) % kRing;
  if (s->ring_used[r] && hipEventSynchronize(s->ring_ev[r]) != hipSuccess) return MOE_EHIP;
  char* h = s->ring + (size_t)r * s->row_bytes;
  std::memcpy(h, &t->slot_of[(size_t)layer * t->n_ids], (size_t)t->n_ids * sizeof(int32_t));
  std::memcpy(h + s->row_so_bytes, &t->bundles[(size_t)layer * t->n_slots],
              (size_t)t->n_slots * sizeof(moe_bundle));
  char* dev = static_cast<char*>(t->dev);
  if (hipMemcpyAsync(dev + (size_t)layer * t->n_ids * sizeof(int32_t), h,
                     (size_t)t->n_ids * sizeof(int32_t), hipMemcpyHostToDevice, st) != hipSuccess)
    return MOE_EHIP;
  if (hipMemcpyAsync(dev + t->bundles_off + (size_t)layer * t->n_slots * sizeof(moe_bundle),
                     h + s->row_so_bytes, (size_t)t->n_slots * sizeof(moe_bundle),
                     hipMemcpyHostToDevice, st) != hipSuccess)
    return MOE_EHIP;
  if (hipEventRecord(s->ring_ev[r], st) != hipSuccess) return MOE_EHIP;
  s->ring_used[r] = 1;
  return MOE_OK;
}

}  // namespace

namespace {

// Everything but the bundle source: host_bundles is null for the file tier.
int create_common(moe_slot_table* table, const moe_bundle_layout* layout, size_t bundle_bytes,
                  const void* const* host_bundles, void* slot_pool, size_t slot_stride,
                  moe_stager** out) {
  if (!table || !layout || !slot_pool || !out || bundle_bytes == 0 ||
      slot_stride < bundle_bytes || (slot_stride & 255) != 0 || !table->dev)
    return MOE_EINVAL;
  if (!layout_ok(layout, bundle_bytes)) return MOE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(slot_pool) & 255) != 0) return MOE_EALIGN;
  const size_t nh = (size_t)table->n_layers * table->n_ids;
  moe_stager* s = new (std::nothrow) moe_stager;
  if (!s) return MOE_ENOMEM;
  s->table = table;
  s->layout = *layout;
  s->bundle_bytes = bundle_bytes;
  s->slot_stride = slot_stride;
  if (host_bundles) s->host.assign(host_bundles, host_bundles + nh);
  s->pool = static_cast<char*>(slot_pool);
  s->set_ev.resize(table->n_layers);
  s->set_seq.resize(table->n_layers);
  int rc = moe_slot_policy_create(table->n_layers, table->n_ids, table->n_slots, &s->policy);
  if (rc != MOE_OK) {
    delete s;
    return rc;
  }
  s->row_so_bytes = ((size_t)table->n_ids * sizeof(int32_t) + 255) / 256 * 256;
  s->row_bytes = s->row_so_bytes + ((size_t)table->n_slots * sizeof(moe_bundle) + 255) / 256 * 256;
  if (hipHostMalloc(reinterpret_cast<void**>(&s->ring), s->row_bytes * kRing,
                    hipHostMallocDefault) != hipSuccess) {
    s->ring = nullptr;
    moe_stager_destroy(s);
    return MOE_ENOMEM;
  }
  s->ring_ev.assign(kRing, nullptr);
  s->ring_used.assign(kRing, 0);
  for (auto& e : s->ring_ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
      moe_stager_destroy(s);
      return MOE_EHIP;
    }
  // the stager owns every binding of the table: start from empty slots
  std::fill(table->slot_of.begin(), table->slot_of.end(), -1);
  std::fill(table->expert_in.begin(), table->expert_in.end(), -1);
  *out = s;
  return MOE_OK;
}

// Copy one record of the mapped file into a bounce buffer over n threads.
void read_record(const char* src, char* dst, size_t n, int threads) {
  if (threads <= 1 || n < ((size_t)1 << 20)) {
    std::memcpy(dst, src, n);
    return;
  }
  const size_t part = (n / threads + 4095) / 4096 * 4096;
  std::vector<std::thread> th;
  for (int k = 1; k < threads; ++k) {
    const size_t o = part * k;
    if (o >= n) break;
    th.emplace_back([=] { std::memcpy(dst + o, src + o, std::min(part, n - o)); });
  }
  std::memcpy(dst, src, std::min(part, n));
  for (auto& x : th) x.join();
}

// File tier, on the I/O thread: record (layer, e) -> a free bounce buffer ->
// slot `slot` by hipMemcpyAsync on `st`. False if a HIP call failed.
bool copy_record(moe_stager* s, int layer, int e, int slot, hipStream_t st) {
  const moe_slot_table* t = s->table;
  char* dst = s->pool + ((size_t)layer * t->n_slots + slot) * s->slot_stride;
  const int b = s->bounce_next;
  s->bounce_next = (b + 1) % s->n_bounce;
  if (s->bounce_used[b] && hipEventSynchronize(s->bounce_ev[b]) != hipSuccess) return false;
  char* bb = s->bounce + (size_t)b * s->bounce_stride;
  const auto t0 = std::chrono::steady_clock::now();
  read_record(s->map + ((size_t)layer * t->n_ids + e) * s->file_stride, bb, s->bundle_bytes, s->n_io);
  s->read_ns += std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0)
                    .count();
  s->read_bytes += (int64_t)s->bundle_bytes;
  if (hipMemcpyAsync(dst, bb, s->bundle_bytes, hipMemcpyHostToDevice, st) != hipSuccess ||
      hipEventRecord(s->bounce_ev[b], st) != hipSuccess)
    return false;
  s->bounce_used[b] = 1;
  return true;
}

void io_loop(moe_stager* s) {
  (void)hipSetDevice(s->device);
  for (;;) {
    moe_stager::IoJob j;
    {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv_job.wait(lk, [&] { return s->stop || !s->jobs.empty(); });
      if (s->jobs.empty()) return;  // stopped, every queued set issued
      j = std::move(s->jobs.front());
      s->jobs.pop_front();
    }
    bool ok = !s->failed.load();
    for (size_t i = 0; ok && 2 * i < j.cp.size(); ++i) ok = copy_record(s, j.layer, j.cp[2 * i], j.cp[2 * i + 1], j.st);
    if (ok && j.ev && hipEventRecord(j.ev, j.st) != hipSuccess) ok = false;
    {
      std::lock_guard<std::mutex> lk(s->mu);
      if (!ok) s->failed = true;
      s->issued = j.seq + 1;
    }
    s->cv_issued.notify_all();
  }
}

}  // namespace

int moe_stager_create(moe_slot_table* table, const moe_bundle_layout* layout, size_t bundle_bytes,
                      const void* const* host_bundles, void* slot_pool, size_t slot_stride,
                      moe_stager** out) {
  if (!table || !host_bundles) return MOE_EINVAL;
  const size_t nh = (size_t)table->n_layers * table->n_ids;
  for (size_t i = 0; i < nh; ++i)
    if (!host_bundles[i]) return MOE_EINVAL;
  return create_common(table, layout, bundle_bytes, host_bundles, slot_pool, slot_stride, out);
}

int moe_stager_create_file(moe_slot_table* table, const moe_bundle_layout* layout,
                           size_t bundle_bytes, const char* path, size_t file_stride, int n_bounce,
                           int n_io, void* slot_pool, size_t slot_stride, moe_stager** out) {
  if (!table || !path || !out || file_stride < bundle_bytes || n_bounce < 1 || n_bounce > 16 ||
      n_io < 1 || n_io > 16)
    return MOE_EINVAL;
  const int fd = open(path, O_RDONLY | O_CLOEXEC);
  if (fd < 0) return MOE_EINVAL;
  struct stat st;
  const size_t need = (size_t)table->n_layers * table->n_ids * file_stride;
  if (fstat(fd, &st) != 0 || (size_t)st.st_size < need) {
    close(fd);
    return MOE_EINVAL;
  }
  void* m = mmap(nullptr, need, PROT_READ, MAP_SHARED, fd, 0);
  if (m == MAP_FAILED) {
    close(fd);
    return MOE_ENOMEM;
  }
  moe_stager* s = nullptr;
  int rc = create_common(table, layout, bundle_bytes, nullptr, slot_pool, slot_stride, &s);
  if (rc != MOE_OK) {
    munmap(m, need);
    close(fd);
    return rc;
  }
  s->fd = fd;
  s->map = static_cast<const char*>(m);
  s->map_bytes = need;
  s->file_stride = file_stride;
  s->n_bounce = n_bounce;
  s->n_io = n_io;
  s->bounce_stride = (bundle_bytes + 4095) / 4096 * 4096;
  if (hipHostMalloc(reinterpret_cast<void**>(&s->bounce), s->bounce_stride * n_bounce,
                    hipHostMallocDefault) != hipSuccess) {
    s->bounce = nullptr;
    moe_stager_destroy(s);
    return MOE_ENOMEM;
  }
  s->bounce_ev.assign(n_bounce, nullptr);
  s->bounce_used.assign(n_bounce, 0);
  for (auto& e : s->bounce_ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
      moe_stager_destroy(s);
      return MOE_EHIP;
    }
  if (hipGetDevice(&s->device) != hipSuccess) {
    moe_stager_destroy(s);
    return MOE_EHIP;
  }
  try {
    s->io = std::thread(io_loop, s);
  } catch (...) {
    moe_stager_destroy(s);
    return MOE_ENOMEM;
  }
  *out = s;
  return MOE_OK;
}

int moe_stager_io_stats(const moe_stager* s, int64_t* read_ns, int64_t* read_bytes) {
  if (!s || !read_ns || !read_bytes) return MOE_EINVAL;
  *read_ns = s->read_ns.load();
  *read_bytes = s->read_bytes.load();
  return MOE_OK;
}

int moe_stager_destroy(moe_stager* s) {
  if (!s) return MOE_OK;
  if (s->io.joinable()) {  // the I/O thread issues every queued set, then leaves
    {
      std::lock_guard<std::mutex> lk(s->mu);
      s->stop = true;
    }
    s->cv_job.notify_all();
    s->io.join();
  }
  for (auto& q : s->set_ev)
    for (hipEvent_t e : q)
      if (e) (void)hipEventDestroy(e);  // null: a set that needed no copy
  for (hipEvent_t e : s->free_ev) (void)hipEventDestroy(e);
  for (hipEvent_t e : s->ring_ev)
    if (e) {
      (void)hipEventSynchronize(e);
      (void)hipEventDestroy(e);
    }
  if (s->ring) (void)hipHostFree(s->ring);
  for (hipEvent_t e : s->bounce_ev)
    if (e) {
      (void)hipEventSynchronize(e);
      (void)hipEventDestroy(e);
    }
  if (s->bounce) (void)hipHostFree(s->bounce);
  if (s->map) munmap(const_cast<char*>(s->map), s->map_bytes);
  if (s->fd >= 0) close(s->fd);
  moe_slot_policy_destroy(s->policy);
  delete s;
  return MOE_OK;
}

int moe_stager_stage(moe_stager* s, int layer, const int32_t* experts, int n, void* copy_stream,
                     int32_t* copies) {
  if (!s) return MOE_EINVAL;
  if (s->failed) return MOE_EHIP;
  std::vector<int32_t> cp((size_t)2 * (n > 0 ? n : 1));
  const int nc = policy_stage(s->policy, layer, experts, n, cp.data());
  if (nc < 0) return nc;
  hipStream_t st = static_cast<hipStream_t>(copy_stream);
  moe_slot_table* t = s->table;
  for (int i = 0; i < nc; ++i) {  // mirror the policy's moves into the slot table
    const int e = cp[2 * i], slot = cp[2 * i + 1];
    int32_t* so = &t->slot_of[(size_t)layer * t->n_ids];
    int32_t* ei = &t->expert_in[(size_t)layer * t->n_slots];
    if (ei[slot] >= 0) so[ei[slot]] = -1;
    so[e] = slot;
    ei[slot] = e;
    t->bundles[(size_t)layer * t->n_slots + slot] = slot_bundle(s, layer, slot);
  }
  // A set with no copy needs no wait: each of its experts was copied for an
  // earlier set of the layer, whose use (first, in FIFO order) waits for it.
  hipEvent_t ev = nullptr;
  if (nc > 0 && !(ev = take_event(s))) {
    s->failed = true;  // the policy and the table already hold the set
    return MOE_EHIP;
  }
  int rc = MOE_OK;
  if (nc > 0) rc = push_rows(s, layer, st);
  if (s->map) {  // file tier: the I/O thread reads the records and issues the copies
    uint64_t seq = kNoJob;
    if (rc == MOE_OK && nc > 0) {
      std::lock_guard<std::mutex> lk(s->mu);
      seq = s->next_seq++;
      s->jobs.push_back(moe_stager::IoJob{layer, std::vector<int32_t>(cp.begin(), cp.begin() + 2 * nc), ev, st, seq});
    }
    if (seq != kNoJob) s->cv_job.notify_one();
    s->set_ev[layer].push_back(ev);
    s->set_seq[layer].push_back(seq);
  } else {
    for (int i = 0; i < nc && rc == MOE_OK; ++i) {
      const int e = cp[2 * i], slot = cp[2 * i + 1];
      char* dst = s->pool + ((size_t)layer * t->n_slots + slot) * s->slot_stride;
      if (hipMemcpyAsync(dst, s->host[(size_t)layer * t->n_ids + e], s->bundle_bytes, hipMemcpyHostToDevice,
                         st) != hipSuccess)
        rc = MOE_EHIP;
    }
    if (rc == MOE_OK && ev && hipEventRecord(ev, st) != hipSuccess) rc = MOE_EHIP;
    s->set_ev[layer].push_back(ev);
  }
  if (rc != MOE_OK) {
    s->failed = true;
    return rc;
  }
  if (copies) std::memcpy(copies, cp.data(), (size_t)2 * nc * sizeof(int32_t));
  s->stats.stages += 1;
  s->stats.copies += nc;
  s->stats.bytes += (int64_t)nc * (int64_t)s->bundle_bytes;
  return nc;
}

int moe_stager_use(moe_stager* s, int layer, const int32_t* experts, int n, void* compute_stream,
                   int32_t* slots) {
  if (!s) return MOE_EINVAL;
  if (s->failed) return MOE_EHIP;
  const int rc = policy_use(s->policy, layer, experts, n, slots);
  if (rc != MOE_OK) return rc;
  hipEvent_t ev = s->set_ev[layer].front();
  s->set_ev[layer].pop_front();
  if (s->map) {  // the set's copies must have been issued (its event recorded)
    const uint64_t seq = s->set_seq[layer].front();
    s->set_seq[layer].pop_front();
    if (seq != kNoJob) {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv_issued.wait(lk, [&] { return s->issued > seq || s->failed; });
      if (s->failed) return MOE_EHIP;
    }
  }
  hipError_t e = hipSuccess;
  if (ev) {
    e = hipStreamWaitEvent(static_cast<hipStream_t>(compute_stream), ev, 0);
    s->free_ev.push_back(ev);
  }
  s->stats.uses += 1;
  return e == hipSuccess ? MOE_OK : MOE_EHIP;
}

int moe_stager_release(moe_stager* s, int layer) {
  if (!s) return MOE_EINVAL;
  return policy_release(s->policy, layer);
}

int moe_stager_stats_get(const moe_stager* s, moe_stager_stats* out) {
  if (!s || !out) return MOE_EINVAL;
  *out = s->stats;
  return MOE_OK;
}
