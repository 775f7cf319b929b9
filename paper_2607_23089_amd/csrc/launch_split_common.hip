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
};
SplitState g_split[kMaxDevices];

constexpr size_t kSplitWorkspaceBytes = (size_t)kSplitMaxBlocks * 32 + 256;
constexpr size_t kSplitErrorOffset = (size_t)kSplitMaxBlocks * 32;

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

int split_begin(hipStream_t stream, uint64_t ntags, SplitTicket* t) {
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
