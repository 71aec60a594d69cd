// Internal helpers shared by the library's translation units (not installed).
#pragma once
#include <cstdarg>
#include <cstdio>
#include <string>

#include "dpool.h"

namespace dpool {

// Record an error message for dp_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Validate a decode shape and report the workspace bytes its launch needs
// (paged_decode.hip): DP_OK, or the error code paged_decode_attention would
// return for the shape, with its message recorded.
int decode_workspace_bytes(const dp_decode_shape* shape, size_t* bytes);

}  // namespace dpool
