// Host-side helpers shared by the library's translation units.
#pragma once

#include <cstdarg>
#include <cstdint>

#include "ooo.h"

namespace ooo {

// Records a thread-local message for ooo_last_error() and returns `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clears the thread-local message; returns OOO_OK.
int ok();

}  // namespace ooo

#define OOO_REQUIRE(cond, status, ...)          \
  do {                                          \
    if (!(cond)) return ::ooo::fail((status), __VA_ARGS__); \
  } while (0)
