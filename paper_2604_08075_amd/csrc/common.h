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

}  // namespace dpool
