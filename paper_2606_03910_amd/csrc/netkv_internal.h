// Declarations shared by the library's translation units (netkv.hip, the
// selection path and the handle; flowsim.hip, the flow-level transfer
// simulation).  Not part of the public interface (include/netkv.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "netkv.h"

// bits of the handle's device error word that the flow simulation sets
constexpr uint32_t kErrFlowBit = 16u;        // invalid flow set
constexpr uint32_t kErrFlowStallBit = 32u;   // an iteration bound was reached

// Record `msg` as the handle's last error and return `st`.
netkv_status netkv_internal_fail(netkv_handle h, netkv_status st, const char *msg);
// Clear the handle's last error (the start of every API call).
void netkv_internal_clear(netkv_handle h);
// The handle's device.
int netkv_internal_device(netkv_handle h);
// The handle's device error word (reported by netkv_sync_errors).
uint32_t *netkv_internal_errword(netkv_handle h);
// A device buffer of the handle for the flow simulation, of at least
// `bytes` (grown on demand, kept until the handle is destroyed).
hipError_t netkv_internal_flow_buffer(netkv_handle h, uint64_t bytes, void **out);
