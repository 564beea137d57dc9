// Range checks of caller-supplied indices read on the device (page-table
// entries, token ids): clamped into range, optionally reported.
#pragma once
#include <hip/hip_runtime.h>

// v clamped into 0 .. n - 1; when it was outside and err (the debug status
// word) is not null, bit (kDevPage / kDevToken) is set in it
__device__ __forceinline__ int checked_index(int v, int n, int* err, int bit) {
  if (v < 0 || v >= n) {
    if (err != nullptr) atomicOr(err, bit);
    v = min(max(v, 0), n - 1);
  }
  return v;
}
