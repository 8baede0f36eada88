// Host-only helpers shared by the C-ABI sources (HIP and plain C++).
#pragma once

#include "rp.h"

namespace rp {
// The value of a C enum field as its caller stored it. The ABI's enums are
// plain ints to a C caller, who may pass any value; in C++ a load of an
// enumeration lvalue outside the enumerators' range is undefined, so host
// code reads the bits as an int and compares those.
template <class E>
inline int enum_bits(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "C enums are int-sized here");
  int v;
  __builtin_memcpy(&v, &e, sizeof v);
  return v;
}

// Records the detail text returned by rp_last_error() on this thread.
rp_status set_error(rp_status st, const char* msg);
void clear_error();
}  // namespace rp
