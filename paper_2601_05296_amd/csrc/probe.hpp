// probe.hpp -- optional per-kernel timing events (see probe.cpp).
#pragma once

#include <hip/hip_runtime.h>

namespace moe {
namespace probe {
bool enabled();
void begin(hipStream_t st);                  // start of an entry point
void mark(const char* name, hipStream_t st); // after a kernel launch
int enable(int capacity);
void disable();
int count();
int dropped();                              // records lost to a full pool
int get(int i, const char** name, float* ms);
}  // namespace probe
}  // namespace moe
