// Per-device state of the single-read split-row form.
//
// The workspace (two 64-bit words per block and row parity, an error count;
// 32 MiB) is allocated and cleared on the first split launch on a device and
// kept until the process ends.  Split launches on one device are ordered
// through `last` (each waits for the previous one, whatever its stream), so
// two launches never use the workspace at the same time.  `last` only orders
// device work against device work, so it is recorded without a system-scope
// fence (and without timing).  Tags are handed
// out from `next_tag`: a launch whose blocks process at most n rows each uses
// tags tag0 .. tag0 + n - 1, so a tag is never reused while the workspace may
// still hold it; when the 32-bit tag space runs out the workspace is cleared
// again and tags restart at 1.
//
// Launches recorded under stream capture cannot take tags from the host (a
// graph replays the recorded arguments), so each gets a private slice of a
// per-device capture region (64 MiB, allocated and cleared with the shared
// workspace): a 256-byte header {epoch, tag base} followed by the exchange
// words of at most kCaptureMaxBlocks blocks.  The graph replays the slice's
// epoch kernel before the split kernel; it advances the epoch by the
// launch's n tags and publishes the tag base, epoch + 1, which the kernel
// reads.  Only that one recorded launch ever uses the slice, with the same
// grid and row count at every replay, so every word a replay reads was
// written by that replay or by the one before it, whose tags are the n
// values just below the current ones (modulo 2^32): stale words never match
// and the slice never needs clearing.  Replays of one recorded launch are
// ordered by their stream; graph executables that share a recorded launch
// must not run at the same time.  A slice is never reclaimed: when the
// region is full (or was never created because no single-read launch has run
// outside capture on the device) a captured launch takes the two-pass form.
#include <mutex>

#include "split_launch.hpp"

namespace rowsm {
namespace {

struct SplitState {
  std::mutex mu;
  void* base = nullptr;
  hipEvent_t last = nullptr;
  bool have_last = false;
  uint32_t next_tag = 1;
  char* cap = nullptr;   // capture region
  size_t cap_used = 0;   // bytes handed out as slices
};
SplitState g_split[kMaxDevices];

constexpr size_t kSplitWorkspaceBytes = (size_t)kSplitMaxBlocks * 32 + 256;
constexpr size_t kSplitErrorOffset = (size_t)kSplitMaxBlocks * 32;
constexpr size_t kCaptureRegionBytes = (size_t)64 << 20;
constexpr size_t kSliceHeaderBytes = 256;

size_t slice_bytes(int64_t blocks) {
  return (kSliceHeaderBytes + (size_t)blocks * 32 + 255) / 256 * 256;
}

// Advances a captured launch's epoch by its tag count and publishes the tag
// base of this replay (hdr[0] epoch, hdr[1] tag base).
__global__ void split_epoch_kernel(uint32_t* hdr, uint32_t ntags) {
  if (threadIdx.x == 0) {
    const uint32_t e = __hip_atomic_load(&hdr[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&hdr[1], e + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&hdr[0], e + ntags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

int split_clear(void* p) {
  if (hipMemset(p, 0, kSplitWorkspaceBytes) != hipSuccess) return ROWSM_EHIP;
  return hipDeviceSynchronize() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
}

int split_workspace(SplitState& st, SplitWorkspace* ws) {
  if (!st.base) {
    void* p = nullptr;
    if (hipMalloc(&p, kSplitWorkspaceBytes) != hipSuccess) return ROWSM_EHIP;
    if (split_clear(p) != ROWSM_OK ||
        hipEventCreateWithFlags(&st.last, hipEventDisableTiming | hipEventDisableSystemFence) !=
            hipSuccess) {
      (void)hipFree(p);
      return ROWSM_EHIP;
    }
    st.base = p;
    st.next_tag = 1;
    // The capture region is optional: without it captured launches take the
    // two-pass form.
    void* r = nullptr;
    if (hipMalloc(&r, kCaptureRegionBytes) == hipSuccess) {
      if (hipMemset(r, 0, kCaptureRegionBytes) == hipSuccess &&
          hipDeviceSynchronize() == hipSuccess) {
        st.cap = static_cast<char*>(r);
        st.cap_used = 0;
      } else {
        (void)hipFree(r);
      }
    }
    (void)hipGetLastError();
  }
  char* b = static_cast<char*>(st.base);
  ws->wm = reinterpret_cast<uint64_t*>(b);
  ws->ws = reinterpret_cast<uint64_t*>(b + (size_t)kSplitMaxBlocks * 16);
  ws->error = reinterpret_cast<uint32_t*>(b + kSplitErrorOffset);
  return ROWSM_OK;
}

// Reserve n consecutive tags (n >= 1); clears the workspace when the tag
// space would wrap.
int split_tags(SplitState& st, uint64_t n, uint32_t* tag0) {
  if (n >= 0x80000000ull) return ROWSM_EINVAL;
  if ((uint64_t)st.next_tag + n > 0xffffffffull) {
    if (st.have_last && hipEventSynchronize(st.last) != hipSuccess) return ROWSM_EHIP;
    if (split_clear(st.base) != ROWSM_OK) return ROWSM_EHIP;
    st.next_tag = 1;
  }
  *tag0 = st.next_tag;
  st.next_tag += (uint32_t)n;
  return ROWSM_OK;
}

}  // namespace

int split_begin(const Call& c, uint64_t ntags, SplitTicket* t) {
  if (c.cap_slice) {
    if (ntags >= 0x80000000ull) return ROWSM_EINVAL;
    uint32_t* hdr = reinterpret_cast<uint32_t*>(c.cap_slice);
    uint64_t* words = reinterpret_cast<uint64_t*>(c.cap_slice + kSliceHeaderBytes);
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ROWSM_EHIP;
    t->captured = true;
    t->ws.wm = words;
    t->ws.ws = words + 2 * c.cap_blocks;
    t->ws.error = reinterpret_cast<uint32_t*>(static_cast<char*>(g_split[dev].base) +
                                              kSplitErrorOffset);
    t->ws.dtag = hdr + 1;
    t->tag0 = 0;
    (void)hipGetLastError();
    split_epoch_kernel<<<1, 64, 0, c.st>>>(hdr, (uint32_t)ntags);
    return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  }
  hipStream_t stream = c.st;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ROWSM_EHIP;
  SplitState& st = g_split[dev];
  st.mu.lock();
  int r = split_workspace(st, &t->ws);
  if (r == ROWSM_OK) r = split_tags(st, ntags, &t->tag0);
  if (r == ROWSM_OK && st.have_last && hipStreamWaitEvent(stream, st.last, 0) != hipSuccess)
    r = ROWSM_EHIP;
  if (r != ROWSM_OK) {
    st.mu.unlock();
    return r;
  }
  t->dev = dev;
  return ROWSM_OK;
}

int split_end(SplitTicket* t, hipStream_t stream, bool launched) {
  if (t->captured) return ROWSM_OK;
  SplitState& st = g_split[t->dev];
  int r = ROWSM_OK;
  if (launched) {
    if (hipEventRecord(st.last, stream) == hipSuccess) st.have_last = true;
    else r = ROWSM_EHIP;
  }
  st.mu.unlock();
  t->dev = -1;
  return r;
}

int split_capture_reserve(int64_t blocks, char** slice) {
  int dev = 0;
  if (blocks < 1 || blocks > kCaptureMaxBlocks) return ROWSM_EINVAL;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ROWSM_EINVAL;
  SplitState& st = g_split[dev];
  std::lock_guard<std::mutex> lock(st.mu);
  const size_t need = slice_bytes(blocks);
  if (!st.cap || st.cap_used + need > kCaptureRegionBytes) return ROWSM_EINVAL;
  *slice = st.cap + st.cap_used;
  st.cap_used += need;
  return ROWSM_OK;
}

int64_t split_wait_failures_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ROWSM_EHIP;
  SplitState& st = g_split[dev];
  std::lock_guard<std::mutex> lock(st.mu);
  if (!st.base) return 0;  // no split launch on this device yet
  if (st.have_last && hipEventSynchronize(st.last) != hipSuccess) return ROWSM_EHIP;
  uint32_t n = 0;
  if (hipMemcpy(&n, static_cast<const char*>(st.base) + kSplitErrorOffset, sizeof(n),
                hipMemcpyDeviceToHost) != hipSuccess)
    return ROWSM_EHIP;
  return (int64_t)n;
}

}  // namespace rowsm
