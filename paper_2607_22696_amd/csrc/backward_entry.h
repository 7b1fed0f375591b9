// Argument checks of the 3D-DSA backward entry points (shared by the caller-workspace entry
// points and the one that runs in the library's fixed scratch buffer).
#pragma once

#include <stddef.h>

#include "dsa3d.h"
#include "dsa3d_internal.h"

namespace dsa3d {

struct BackwardArgs {
  const void *q, *k, *v;
  const float* offsets;
  const void* out;  // optional, not read
  const float* lse;
  const void* dout;
  float *dq, *dk, *dv, *d_offsets;
};

// Checks a backward call and fills the kernel geometry.  scratch_limit == 0: `workspace` is the
// caller's (NULL, too small, misaligned or overlapping arguments are errors); otherwise the
// workspace is the library's fixed scratch buffer of scratch_limit bytes and a problem that
// needs more returns DSA3D_ERR_SCRATCH.  Never touches the device.
dsa3d_status check_backward_call(const dsa3d_desc* desc, const BackwardArgs& a,
                                 const void* workspace, size_t workspace_bytes,
                                 size_t scratch_limit, Geometry* g);

}  // namespace dsa3d
