// Optional per-launch event timing used by hydra_profile_start / hydra_profile_stop.
#pragma once
#include <hip/hip_runtime.h>

namespace hydra {
// Returns a token (or -1 when not recording) after recording a start event on `stream`.
int prof_begin(const char* kernel, hipStream_t stream);
// Records the end event for `token` on `stream` (no-op for -1).
void prof_end(int token, hipStream_t stream);
}  // namespace hydra
