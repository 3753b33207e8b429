// Host-side helpers shared by the translation units of libbitsmoe.
#pragma once

#include <cstddef>
#include <cstdint>
#include <initializer_list>
#include <string>

#include "bitsmoe.h"

namespace bitsmoe {

// Records `msg` as the calling thread's last error and returns `st`.
bitsmoe_status fail(bitsmoe_status st, const std::string& msg);
// Clears the calling thread's last error; returns BITSMOE_OK.
bitsmoe_status ok();

// Named scratch regions.  Each is a grow-only device buffer per device.
enum ScratchSlot : int {
  kScratchA = 0,     // operand staging (transposes, bf16 splits)
  kScratchB = 1,     // second operand staging
  kScratchPart = 2,  // split-K / row partials
  kScratchD = 3,     // score: bf16 error rows
  kScratchMisc = 4,  // small tables
  kScratchCount = 5
};

// Returns a device buffer of at least `bytes` bytes for `slot` on the
// current device.  Growing synchronizes `stream` first (calls on a device
// are stream-ordered, so no queued work still reads the old buffer).
// Returns nullptr after recording ERR_NOMEM / ERR_DEVICE.
void* scratch(int slot, size_t bytes, void* stream, bitsmoe_status* st);

// HIP error -> status with a message naming `what`.
bitsmoe_status device_error(const char* what, int hip_err);

// Compute units of the current device (cached per device; 256 if the query
// fails).
int device_cus();

// Records HIP events around a kernel launch when timing is enabled
// (bitsmoe_timing); construct right before the launch, destroy right after.
// A null name records nothing.
class KernelTimer {
 public:
  KernelTimer(const char* name, void* stream);
  ~KernelTimer();
 private:
  const char* name_;
  void* stream_;
  void* start_ = nullptr;
};

// True when every pointer is 16-byte aligned (the kernels use 16-byte
// vector accesses on device buffers).
inline bool aligned16(std::initializer_list<const void*> ptrs) {
  for (const void* p : ptrs)
    if (reinterpret_cast<uintptr_t>(p) % 16 != 0) return false;
  return true;
}

inline bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

}  // namespace bitsmoe
