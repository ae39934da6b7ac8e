// SSD -> DRAM tier (Sec. 5.4 "Pattern-Aware Preloading for SSD", Fig. 8):
// every layer's neuron records live in a file; a two-level DRAM cache keeps
// the first `fixed` layers in a fixed area (loaded once, never evicted) and
// the others in a dynamic area of layer slots; a loader thread reads whole
// layers ahead of the layer being used.
//
// Decisions are made under the cache's lock when a layer is acquired, in a
// fixed order, so they depend only on the order of acquires, never on how
// fast the loads go: for the acquired layer l the window W(l) = l .. l + a
// (mod L) is made resident in order (l first, the consumer waits for it);
// a missing layer takes the lowest empty slot, else the slot whose layer is
// outside W(l), not held by a consumer, and used furthest in the future in
// the cyclic layer order, the largest (layer - l) mod L (if its own load is
// still running, the acquire waits for it). A look-ahead load with no slot
// to give up is skipped.
//
// A slot's bytes may still be read by GPU fills already enqueued; the
// consumer attaches a HIP event when it releases the slot, and the loader
// waits for every such event before it writes a new layer into the slot.
#include <errno.h>
#include <fcntl.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <chrono>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

#include "m2c_internal.h"

struct m2c_dram {
  m2c_dram_desc desc;
  int fd = -1;
  bool direct = false;  // reads bypass the page cache (O_DIRECT)
  int64_t read_bytes = 0;  // per layer: layer_bytes rounded up to 4096
  std::vector<int64_t> offsets;
  std::vector<uint8_t*> fixed_buf;  // [fixed]
  struct Slot {
    uint8_t* buf = nullptr;
    int layer = -1;
    bool ready = false;
    int pins = 0;                       // consumers between acquire and release
    std::vector<hipEvent_t> pending;    // GPU readers to wait for before a reload
  };
  std::vector<Slot> slots;
  std::vector<int> where;  // layer -> slot, -1 not resident, -2 fixed area
  struct Job {
    int slot, layer;
  };
  std::deque<Job> queue;
  std::vector<hipEvent_t> free_events;
  std::mutex mu;
  std::condition_variable cv;  // queue / readiness / releases
  std::thread loader;
  bool stop = false;
  int io_error = 0;  // errno of a failed read (reported by the next acquire)
  int refs = 0;      // layers bound to the cache
  m2c_dram_stats st{};
  std::vector<int32_t> log_loaded, log_evicted;
  uint8_t* bounce = nullptr;  // direct reads land here first (pinned pages refuse O_DIRECT)
};

constexpr int64_t kBounceBytes = 32 << 20;

namespace {

bool pinned(const m2c_dram_desc& d) { return (d.flags & M2C_DRAM_HOST_MEMORY) == 0; }

uint8_t* alloc_buf(const m2c_dram_desc& d, int64_t bytes) {
  if (pinned(d)) {
    void* p = nullptr;
    if (hipHostMalloc(&p, (size_t)bytes, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    return (uint8_t*)p;
  }
  return (uint8_t*)aligned_alloc(4096, (size_t)bytes);
}

void free_buf(const m2c_dram_desc& d, uint8_t* p) {
  if (!p) return;
  if (pinned(d))
    (void)hipHostFree(p);
  else
    free(p);
}

// Reads layer `layer` into `buf`; returns 0 or an errno value. Direct reads
// go through the bounce buffer: the kernel cannot pin hipHostMalloc pages
// for O_DIRECT (EFAULT), and the copy out of the bounce buffer is much
// faster than the device.
int read_layer(m2c_dram* D, int layer, uint8_t* buf) {
  int64_t off = D->offsets[layer], done = 0;
  const int64_t want = D->direct ? D->read_bytes : D->desc.layer_bytes;
  const int64_t max_chunk = D->direct ? kBounceBytes : (64 << 20);
  while (done < want) {
    const int64_t chunk = want - done < max_chunk ? want - done : max_chunk;
    uint8_t* dst = D->direct ? D->bounce : buf + done;
    const ssize_t r = pread(D->fd, dst, (size_t)chunk, off + done);
    if (r < 0) {
      if (errno == EINTR) continue;
      return errno;
    }
    if (r == 0) {
      // past the end of the file: only the padding of the last layer may be missing
      if (done >= D->desc.layer_bytes) break;
      return EIO;
    }
    if (D->direct) {
      // the buffer holds read_bytes; copy only what belongs to the layer
      const int64_t keep = done + r <= D->read_bytes ? r : D->read_bytes - done;
      memcpy(buf + done, D->bounce, (size_t)keep);
    }
    done += r;
  }
  return 0;
}

void loader_main(m2c_dram* D) {
  if (pinned(D->desc)) (void)hipSetDevice(D->desc.device);
  std::unique_lock<std::mutex> lk(D->mu);
  for (;;) {
    D->cv.wait(lk, [&] { return D->stop || !D->queue.empty(); });
    if (D->stop) return;
    const m2c_dram::Job job = D->queue.front();
    D->queue.pop_front();
    m2c_dram::Slot& s = D->slots[job.slot];
    std::vector<hipEvent_t> waits;
    waits.swap(s.pending);
    uint8_t* buf = s.buf;
    lk.unlock();
    for (hipEvent_t e : waits) (void)hipEventSynchronize(e);
    const auto t0 = std::chrono::steady_clock::now();
    const int err = read_layer(D, job.layer, buf);
    const double secs = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    lk.lock();
    for (hipEvent_t e : waits) D->free_events.push_back(e);
    D->st.read_seconds += secs;
    if (err) {
      D->io_error = err;
    } else {
      D->st.loads++;
      D->st.bytes_read += D->desc.layer_bytes;
    }
    s.ready = true;  // even on error: the next acquire reports io_error instead of waiting forever
    D->cv.notify_all();
  }
}

// Makes layer m resident or queued for the window of layer l (lock held).
// Returns false if the layer could not be placed.
// A victim that is still loading is waited for (lk is the cache's lock), not
// passed over, so that the choice does not depend on how fast loads go.
bool ensure(m2c_dram* D, std::unique_lock<std::mutex>& lk, int l, int m) {
  const int L = D->desc.n_layers, a = D->desc.lookahead;
  for (;;) {
    if (D->where[m] != -1) return true;
    int pick = -1;
    for (int q = 0; q < (int)D->slots.size(); ++q)
      if (D->slots[q].layer < 0) {
        pick = q;
        break;
      }
    int old = -1;
    if (pick < 0) {
      int best = -1;
      for (int q = 0; q < (int)D->slots.size(); ++q) {
        const m2c_dram::Slot& s = D->slots[q];
        if (s.pins > 0) continue;
        const int dist = ((s.layer - l) % L + L) % L;
        if (dist <= a) continue;  // inside the window
        if (dist > best) {
          best = dist;
          pick = q;
        }
      }
      if (pick < 0) return false;
      if (!D->slots[pick].ready) {  // its load ends on its own (ready is set even on error)
        D->cv.wait(lk);
        continue;
      }
      old = D->slots[pick].layer;
      D->where[old] = -1;
      D->st.evictions++;
    }
    m2c_dram::Slot& s = D->slots[pick];
    s.layer = m;
    s.ready = false;
    D->where[m] = pick;
    D->queue.push_back({pick, m});
    D->log_loaded.push_back(m);
    D->log_evicted.push_back(old);
    D->cv.notify_all();
    return true;
  }
}

}  // namespace

namespace m2c {

// Blocks until layer `layer` is in DRAM, holds it, and returns its bytes and
// slot (-1 for the fixed area). Lock not held on entry.
m2c_status dram_acquire(m2c_dram* D, int layer, const uint8_t** data, int* slot) {
  std::unique_lock<std::mutex> lk(D->mu);
  if (D->io_error)
    return api_fail(M2C_ERR_HIP, "reading the layer file failed: %s", strerror(D->io_error));
  D->st.acquires++;
  const int L = D->desc.n_layers;
  const bool hit = D->where[layer] != -1 &&
                   (D->where[layer] == -2 || D->slots[D->where[layer]].ready);
  if (hit) D->st.hits++;
  const auto t0 = std::chrono::steady_clock::now();
  for (;;) {
    // the layer in use first, then the look-ahead in order
    const bool placed = ensure(D, lk, layer, layer);
    for (int j = 1; j <= D->desc.lookahead; ++j) ensure(D, lk, layer, (layer + j) % L);
    if (placed) break;
    D->cv.wait(lk);  // every slot is held: wait for a release
  }
  const int w = D->where[layer];
  if (w == -2) {
    *data = D->fixed_buf[layer];
    *slot = -1;
  } else {
    m2c_dram::Slot& s = D->slots[w];
    s.pins++;
    D->cv.wait(lk, [&] { return s.ready; });
    *data = s.buf;
    *slot = w;
  }
  D->st.wait_seconds +=
      std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  if (D->io_error) {
    if (w >= 0) D->slots[w].pins--;
    return api_fail(M2C_ERR_HIP, "reading the layer file failed: %s", strerror(D->io_error));
  }
  return M2C_OK;
}

// Gives up a hold from dram_acquire; `reader` (may be null) is a HIP event
// after the last GPU read of the slot's bytes.
void dram_release(m2c_dram* D, int slot, hipEvent_t reader) {
  std::lock_guard<std::mutex> lk(D->mu);
  if (slot < 0) return;
  m2c_dram::Slot& s = D->slots[slot];
  if (reader) s.pending.push_back(reader);
  if (s.pins > 0) s.pins--;
  D->cv.notify_all();
}

// An event from the cache's pool (created on first use).
hipEvent_t dram_event(m2c_dram* D) {
  {
    std::lock_guard<std::mutex> lk(D->mu);
    if (!D->free_events.empty()) {
      hipEvent_t e = D->free_events.back();
      D->free_events.pop_back();
      return e;
    }
  }
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  return e;
}

int64_t dram_layer_bytes(const m2c_dram* D) { return D->desc.layer_bytes; }
int dram_layers(const m2c_dram* D) { return D->desc.n_layers; }
int dram_device(const m2c_dram* D) { return D->desc.device; }
bool dram_pinned(const m2c_dram* D) { return pinned(D->desc); }
void dram_ref(m2c_dram* D, int delta) {
  std::lock_guard<std::mutex> lk(D->mu);
  D->refs += delta;
}

}  // namespace m2c

extern "C" {

m2c_status m2c_dram_create(const m2c_dram_desc* desc, const char* path, const int64_t* offsets,
                           m2c_dram** out) {
  if (!desc || !path || !offsets || !out) return m2c::api_fail(M2C_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  const m2c_dram_desc& d = *desc;
  if (d.n_layers < 1 || d.fixed_layers < 0 || d.fixed_layers > d.n_layers || d.lookahead < 1 ||
      d.dynamic_slots < 0 || d.layer_bytes <= 0)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "bad descriptor (layers %d, fixed %d, slots %d, "
                         "lookahead %d, layer_bytes %lld)", d.n_layers, d.fixed_layers,
                         d.dynamic_slots, d.lookahead, (long long)d.layer_bytes);
  if (d.fixed_layers < d.n_layers && d.dynamic_slots < d.lookahead + 1)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "dynamic_slots %d: at least lookahead + 1 = %d are "
                         "needed", d.dynamic_slots, d.lookahead + 1);
  if (d.flags & ~(M2C_DRAM_HOST_MEMORY | M2C_DRAM_DIRECT_IO))
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "flags 0x%x: unknown bits", d.flags);
  for (int l = 0; l < d.n_layers; ++l)
    if (offsets[l] < 0 || offsets[l] % 4096)
      return m2c::api_fail(M2C_ERR_INVALID_ARG, "offset of layer %d (%lld) must be a multiple "
                           "of 4096", l, (long long)offsets[l]);
  m2c_dram* D = new (std::nothrow) m2c_dram();
  if (!D) return m2c::api_fail(M2C_ERR_OUT_OF_MEMORY, "host allocation failed");
  D->desc = d;
  D->read_bytes = (d.layer_bytes + 4095) / 4096 * 4096;
  D->offsets.assign(offsets, offsets + d.n_layers);
  if (pinned(d) && hipSetDevice(d.device) != hipSuccess) {
    (void)hipGetLastError();
    delete D;
    return m2c::api_fail(M2C_ERR_HIP, "hipSetDevice(%d) failed", d.device);
  }
  if (d.flags & M2C_DRAM_DIRECT_IO) {
    D->fd = open(path, O_RDONLY | O_DIRECT);
    D->direct = D->fd >= 0;
  }
  if (D->fd < 0) D->fd = open(path, O_RDONLY);
  if (D->fd < 0) {
    const int e = errno;
    delete D;
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "open(%s): %s", path, strerror(e));
  }
  if (D->direct) {
    D->bounce = (uint8_t*)aligned_alloc(4096, (size_t)kBounceBytes);
    if (!D->bounce) {
      close(D->fd);
      delete D;
      return m2c::api_fail(M2C_ERR_OUT_OF_MEMORY, "DRAM cache: bounce buffer allocation failed");
    }
  } else {
    (void)posix_fadvise(D->fd, 0, 0, POSIX_FADV_DONTNEED);
  }
  D->st.direct_io = D->direct ? 1 : 0;
  D->where.assign(d.n_layers, -1);
  m2c_status rc = M2C_OK;
  for (int l = 0; l < d.fixed_layers && rc == M2C_OK; ++l) {
    uint8_t* b = alloc_buf(d, D->read_bytes);
    if (!b) {
      rc = m2c::api_fail(M2C_ERR_OUT_OF_MEMORY, "DRAM cache: fixed area allocation failed");
      break;
    }
    D->fixed_buf.push_back(b);
    const int err = read_layer(D, l, b);
    if (err) rc = m2c::api_fail(M2C_ERR_HIP, "reading layer %d: %s", l, strerror(err));
    D->where[l] = -2;
    D->st.fixed_bytes += d.layer_bytes;
  }
  if (rc == M2C_OK && d.fixed_layers < d.n_layers) {
    D->slots.resize(d.dynamic_slots);
    for (auto& s : D->slots) {
      s.buf = alloc_buf(d, D->read_bytes);
      if (!s.buf) {
        rc = m2c::api_fail(M2C_ERR_OUT_OF_MEMORY, "DRAM cache: dynamic area allocation failed");
        break;
      }
    }
  }
  if (rc != M2C_OK) {
    m2c_dram_destroy(D);
    return rc;
  }
  D->loader = std::thread(loader_main, D);
  *out = D;
  return M2C_OK;
}

m2c_status m2c_dram_destroy(m2c_dram* D) {
  if (!D) return M2C_OK;
  {
    std::lock_guard<std::mutex> lk(D->mu);
    if (D->refs > 0)
      return m2c::api_fail(M2C_ERR_STATE, "%d layers still read from this DRAM cache", D->refs);
    D->stop = true;
    D->cv.notify_all();
  }
  if (D->loader.joinable()) D->loader.join();
  for (auto& s : D->slots) {
    for (hipEvent_t e : s.pending) (void)hipEventSynchronize(e);
    for (hipEvent_t e : s.pending) D->free_events.push_back(e);
    free_buf(D->desc, s.buf);
  }
  for (uint8_t* b : D->fixed_buf) free_buf(D->desc, b);
  for (hipEvent_t e : D->free_events) (void)hipEventDestroy(e);
  if (D->fd >= 0) close(D->fd);
  free(D->bounce);
  delete D;
  return M2C_OK;
}

m2c_status m2c_dram_acquire(m2c_dram* D, int32_t layer, const uint8_t** data) {
  if (!D || !data) return m2c::api_fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (layer < 0 || layer >= D->desc.n_layers)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, D->desc.n_layers);
  int slot = -1;
  return m2c::dram_acquire(D, layer, data, &slot);
}

m2c_status m2c_dram_release(m2c_dram* D, int32_t layer) {
  if (!D) return m2c::api_fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (layer < 0 || layer >= D->desc.n_layers)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, D->desc.n_layers);
  int slot;
  {
    std::lock_guard<std::mutex> lk(D->mu);
    slot = D->where[layer];
    if (slot == -1 || (slot >= 0 && D->slots[slot].pins == 0))
      return m2c::api_fail(M2C_ERR_STATE, "layer %d is not held", layer);
  }
  m2c::dram_release(D, slot, nullptr);
  return M2C_OK;
}

m2c_status m2c_dram_get_stats(m2c_dram* D, m2c_dram_stats* out) {
  if (!D || !out) return m2c::api_fail(M2C_ERR_INVALID_ARG, "NULL argument");
  std::lock_guard<std::mutex> lk(D->mu);
  *out = D->st;
  return M2C_OK;
}

m2c_status m2c_dram_get_log(m2c_dram* D, int32_t* loaded, int32_t* evicted, int32_t capacity,
                            int32_t* count) {
  if (!D || !count) return m2c::api_fail(M2C_ERR_INVALID_ARG, "NULL argument");
  std::lock_guard<std::mutex> lk(D->mu);
  const int n = (int)D->log_loaded.size();
  *count = n;
  for (int i = 0; i < n && i < capacity; ++i) {
    if (loaded) loaded[i] = D->log_loaded[i];
    if (evicted) evicted[i] = D->log_evicted[i];
  }
  return M2C_OK;
}

}  // extern "C"
