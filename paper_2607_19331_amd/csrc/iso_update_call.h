// iso_update's body with a pluggable workspace source (internal): the public iso_update passes the
// caller's workspace, iso_update_noalloc a fixed block of static device memory.
#pragma once

#include <stddef.h>

#include "iso.h"

namespace iso {

struct WsSource {
  void* ws = nullptr;      // the caller's workspace (when acquire is null)
  size_t bytes = 0;
  // Hands out a workspace of at least `need` bytes or rejects the call; also switches off the
  // profiling events (their creation allocates).
  iso_status (*acquire)(size_t need, void** ws, size_t* bytes) = nullptr;
};

iso_status update_call(const iso_tensor* t, int n_t, int K, int dt, const iso_update_args* a,
                       const WsSource& src, void* stream);

}  // namespace iso
