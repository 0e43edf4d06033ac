// Internal helpers shared by the library's translation units.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "rnnbkt.h"

namespace rnnbkt {

// Thread-local last-error text behind rnnbkt_last_error().
void set_error(const char* fmt, ...);
void clear_error();

}  // namespace rnnbkt

#define RNNBKT_REQUIRE(cond, code, ...)   \
  do {                                    \
    if (!(cond)) {                        \
      ::rnnbkt::set_error(__VA_ARGS__);   \
      return (code);                      \
    }                                     \
  } while (0)
