// Exchange workspaces of the forms whose blocks share a row (the single-read
// split forms, and the two-pass forms with several blocks per row).
//
// A launch takes a region of 32 bytes per block (two parities of a max and a
// sum word, split_row.hpp) and a run of 32-bit tags from a ring of words per
// device.  The first ring is the static device array `exchange_words` (64 MiB
// per device, zero from the moment the library's device code is loaded, so
// no call allocates, clears or waits for anything to use it); its address is
// looked up once per device (hipGetSymbolAddress, with that device current)
// and host code never passes the array's own name to a kernel.  A ring's tags
// count up from 1, and once they pass 2^30 the ring is retired (kept, unused)
// and replaced by a 64 MiB allocation cleared on a private stream of the
// library that the host waits for (that stream holds nothing else, so no
// caller's work is waited for): a ring never sees two launches with the same
// tag, so a word it holds that carries a launch's tag was written by that
// launch.  Regions are handed out in turn by an atomic cursor, so launches in
// flight together on any streams take disjoint regions unless the ring wraps
// while one of them is still waiting to run.  No launch waits for or is
// ordered after another.  Launches in flight together have different tags,
// so words of another launch that shares the region after a wrap cost at most
// waits that give up and a recomputation, never a wrong result.
//
// Stream capture: a graph replays the region and the tags recorded at
// capture, so a captured launch is preceded by a recorded kernel that clears
// its region; every replay then starts from cleared words.  Graph
// executables that contain the same captured launch must not run at the same
// time (they would share tags as well as words).  A ring is never renewed
// under capture.
#include <atomic>
#include <mutex>

#include "split_launch.hpp"

namespace rowsm {

constexpr int64_t kRingBlocks = (int64_t)1 << 21;  // 64 MiB per ring
constexpr int64_t kRingHeaderWords = 32;           // 256 bytes: the give-up counter
static_assert(kSplitMaxBlocks <= kRingBlocks / 2, "a launch takes at most half the ring");
static __device__ __align__(256) uint64_t exchange_words[kRingHeaderWords + 4 * kRingBlocks];

// The workspace of rowsm_forward_noalloc(), for callers that cannot allocate:
// the static device array `scratch` (4 MiB per device and a 256-byte header
// whose first word counts its give-ups), never replaced, so its tags wrap
// around and every launch on it first clears its own region with a kernel on
// its stream.  Every call on a device shares it; calls in flight together
// take different regions unless it wraps, and different tags, so overlapping
// calls can slow each other down (a block whose peer's words were cleared or
// overwritten recomputes them) but not change each other's results.
constexpr int64_t kScratchBlocks = (int64_t)1 << 17;
static __device__ __align__(256) uint64_t scratch[kRingHeaderWords + 4 * kScratchBlocks];

namespace {

// A ring is replaced once its tags pass this count (a launch takes at most
// kMaxLaunchTags), so a ring's tags stay below 2^31: unique and never 0 in
// 32 bits.
constexpr uint64_t kRingRenewTag = (uint64_t)1 << 30;
constexpr uint64_t kMaxLaunchTags = (uint64_t)1 << 30;
// Polls before a wait gives up: about 0.1 s at the latency of an agent-scope
// load under streaming traffic.
constexpr uint32_t kDefaultWaitLimit = 1u << 16;

struct Ring {
  uint64_t* words = nullptr;  // device memory, 4 words per block
  int64_t blocks = 0;
  bool clears = false;        // every launch clears its region first (tags wrap)
  std::atomic<int64_t> cursor{0};
  std::atomic<uint64_t> next_tag{1};

  // First block of a region of n <= blocks blocks.
  int64_t take(int64_t n) {
    int64_t old = cursor.load(std::memory_order_relaxed);
    for (;;) {
      const int64_t at = old + n <= blocks ? old : 0;
      if (cursor.compare_exchange_weak(old, at + n, std::memory_order_relaxed)) return at;
    }
  }
  // First of n consecutive tags (1 <= n <= kMaxLaunchTags).  A ring that
  // does not clear keeps them below 2^31 and returns false when they would
  // not be (it is renewed long before, so this needs several launches of
  // about 2^30 rows per block group at once); on a clearing ring they wrap
  // around, skipping runs that would hold 0.
  bool tags(uint64_t n, uint32_t* t0) {
    for (;;) {
      const uint64_t t = next_tag.fetch_add(n, std::memory_order_relaxed);
      if (!clears) {
        if (t + n > ((uint64_t)1 << 31)) return false;
        *t0 = (uint32_t)t;
        return true;
      }
      if ((uint32_t)t != 0 && (t >> 32) == ((t + n - 1) >> 32)) {
        *t0 = (uint32_t)t;
        return true;
      }
    }
  }
};

struct DeviceState {
  std::mutex mu;                     // set-up and renewal of this device's rings
  std::atomic<Ring*> ring{nullptr};  // current ring (retired ones are kept)
  uint32_t* failures = nullptr;      // give-up counter (exchange_words header)
  std::atomic<Ring*> scratch_ring{nullptr};  // the scratch array, once looked up
  uint32_t* scratch_failures = nullptr;      // its give-up counter
};

DeviceState g_dev[kMaxDevices];
std::atomic<uint32_t> g_wait_limit{kDefaultWaitLimit};

__global__ void exchange_clear_kernel(uint64_t* w, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    w[i] = 0;
}

int clear_words(uint64_t* w, int64_t n, hipStream_t st) {
  const int64_t blocks = (n + 255) / 256;
  (void)hipGetLastError();
  exchange_clear_kernel<<<dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, st>>>(w, n);
  return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
}

// A failed query counts as capture.
bool stream_capturing(hipStream_t s) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess) return true;
  return cs != hipStreamCaptureStatusNone;
}

int current_device(DeviceState** d) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ROWSM_EHIP;
  *d = &g_dev[dev];
  return ROWSM_OK;
}

// A fresh ring in place of one whose tags passed kRingRenewTag: an
// allocation cleared on a private stream that the host waits for.  nullptr
// when that fails.
Ring* fresh_ring() {
  hipStream_t s = nullptr;
  void* p = nullptr;
  Ring* fresh = nullptr;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess) {
    if (hipMalloc(&p, (size_t)kRingBlocks * 32) == hipSuccess) {
      const bool cleared = clear_words(static_cast<uint64_t*>(p), 4 * kRingBlocks, s) == ROWSM_OK;
      if (hipStreamSynchronize(s) == hipSuccess && cleared) {
        fresh = new Ring();
        fresh->words = static_cast<uint64_t*>(p);
        fresh->blocks = kRingBlocks;
      } else {
        (void)hipFree(p);
      }
    }
    (void)hipStreamDestroy(s);
  }
  (void)hipGetLastError();
  return fresh;
}

// The current ring of the device: exchange_words (its address looked up on
// first use), or its replacement once the tags pass kRingRenewTag (not under
// capture; when a replacement cannot be made the ring stays, and its launches
// fail once the tags run out).
int device_ring(DeviceState* d, bool capturing, Ring** out) {
  Ring* r = d->ring.load(std::memory_order_acquire);
  if (r && (capturing || r->next_tag.load(std::memory_order_relaxed) <= kRingRenewTag)) {
    *out = r;
    return ROWSM_OK;
  }
  std::lock_guard<std::mutex> lock(d->mu);
  r = d->ring.load(std::memory_order_relaxed);
  if (!r) {
    uint64_t* p = nullptr;
    if (hipGetSymbolAddress(reinterpret_cast<void**>(&p), HIP_SYMBOL(exchange_words)) !=
            hipSuccess ||
        p == nullptr) {
      (void)hipGetLastError();
      return ROWSM_EHIP;
    }
    r = new Ring();
    r->words = p + kRingHeaderWords;
    r->blocks = kRingBlocks;
    d->failures = reinterpret_cast<uint32_t*>(p);
    d->ring.store(r, std::memory_order_release);
  } else if (!capturing && r->next_tag.load(std::memory_order_relaxed) > kRingRenewTag) {
    if (Ring* fresh = fresh_ring()) {
      r = fresh;
      d->ring.store(r, std::memory_order_release);
    }
  }
  *out = r;
  return ROWSM_OK;
}

// The scratch ring of the device: `scratch`, its address looked up on the
// first allocation-free call on the device, with that device current.
int device_scratch(DeviceState* d, Ring** out) {
  Ring* r = d->scratch_ring.load(std::memory_order_acquire);
  if (!r) {
    std::lock_guard<std::mutex> lock(d->mu);
    r = d->scratch_ring.load(std::memory_order_relaxed);
    if (!r) {
      uint64_t* p = nullptr;
      if (hipGetSymbolAddress(reinterpret_cast<void**>(&p), HIP_SYMBOL(scratch)) != hipSuccess ||
          p == nullptr) {
        (void)hipGetLastError();
        return ROWSM_EHIP;
      }
      r = new Ring();
      r->words = p + kRingHeaderWords;
      r->blocks = kScratchBlocks;
      r->clears = true;
      d->scratch_failures = reinterpret_cast<uint32_t*>(p);
      d->scratch_ring.store(r, std::memory_order_release);
    }
  }
  *out = r;
  return ROWSM_OK;
}

}  // namespace

int exchange_ring(const Call& c, ExchangeRing* r) {
  DeviceState* d = nullptr;
  int st = current_device(&d);
  r->capturing = stream_capturing(c.st);
  Ring* ring = nullptr;
  if (st == ROWSM_OK)
    st = c.noalloc ? device_scratch(d, &ring) : device_ring(d, r->capturing, &ring);
  if (st != ROWSM_OK) return st;
  r->ring = ring;
  r->failures = c.noalloc ? d->scratch_failures : d->failures;
  r->max_blocks = c.noalloc ? kScratchBlocks : kSplitMaxBlocks;
  return ROWSM_OK;
}

int exchange_begin(const Call& c, const ExchangeRing& r, int64_t blocks, uint64_t ntags,
                   Exchange* e) {
  if (blocks < 1 || blocks > r.max_blocks || ntags < 1 || ntags > kMaxLaunchTags)
    return ROWSM_EINVAL;
  Ring* ring = static_cast<Ring*>(r.ring);
  uint32_t t0 = 0;
  if (!ring->tags(ntags, &t0)) return ROWSM_EINVAL;
  uint64_t* words = ring->words + 4 * ring->take(blocks);
  if ((r.capturing || ring->clears) && clear_words(words, 4 * blocks, c.st) != ROWSM_OK)
    return ROWSM_EHIP;
  e->ws.words = words;
  e->ws.error = r.failures;
  e->ws.limit = g_wait_limit.load(std::memory_order_relaxed);
  e->tag0 = t0;
  return ROWSM_OK;
}

int64_t split_wait_failures_current_device() {
  DeviceState* d = nullptr;
  if (current_device(&d) != ROWSM_OK) return ROWSM_EHIP;
  const bool ring = d->ring.load(std::memory_order_acquire) != nullptr;
  const bool scr = d->scratch_ring.load(std::memory_order_acquire) != nullptr;
  if (!ring && !scr) return 0;  // no exchange yet
  if (hipDeviceSynchronize() != hipSuccess) return ROWSM_EHIP;
  int64_t total = 0;
  for (uint32_t* counter : {ring ? d->failures : nullptr, scr ? d->scratch_failures : nullptr}) {
    uint32_t n = 0;
    if (counter && hipMemcpy(&n, counter, sizeof(n), hipMemcpyDeviceToHost) != hipSuccess)
      return ROWSM_EHIP;
    total += n;
  }
  return total;
}

int64_t split_set_wait_limit(int64_t polls) {
  uint32_t v = kDefaultWaitLimit;
  if (polls >= 0) v = polls > 0xffffffffll ? 0xffffffffu : (uint32_t)polls;
  return (int64_t)g_wait_limit.exchange(v, std::memory_order_relaxed);
}

}  // namespace rowsm
