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
// events[2 i + 1] after it. ws: the workspace to run in (nullptr: the plan's).
void enqueue(const Plan &p, hipStream_t s, hipEvent_t *events = nullptr, void *ws = nullptr);

// Bytes of the static scratch array of the no-allocation entry point.
constexpr size_t kScratchBytes = SLORR_SCRATCH_BYTES;

// Device address of the static scratch array on the current device (taken
// with hipGetSymbolAddress on the first call per device, then kept).
void *scratch_address();

// Enqueues only the gradient launches (p.grad_launches), reading the state
// (X_T, M, X_0) and the gradient factors a previous enqueue left in the
// workspace.
void enqueue_grad(const Plan &p, hipStream_t s);

// Enqueues the decoupled update W <- W - s G over every matrix (one block per
// element chunk); pointers and steps come from the uploaded call tables.
void enqueue_apply(const Plan &p, hipStream_t s);

}  // namespace slorr
