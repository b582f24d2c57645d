// Kernel enqueue entry of the SLORR library (internal).
#pragma once
#include <hip/hip_runtime.h>

#include <stdexcept>
#include <string>

#include "plan.hpp"

namespace slorr {

struct HipError : std::runtime_error {
  explicit HipError(const std::string &m) : std::runtime_error(m) {}
};

// Enqueue the plan's whole launch schedule on stream s (throws HipError).
// With events != nullptr, events[2 i] is recorded before launch i and
// events[2 i + 1] after it.
void enqueue(const Plan &p, hipStream_t s, hipEvent_t *events = nullptr);

}  // namespace slorr
