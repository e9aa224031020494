// Device-side checks of debug builds.
#pragma once
// Debug builds (SSM_DEBUG defined) check on the device the invariants that the
// host validation promises and that the kernels otherwise rely on or turn into
// NaN rows and skipped writes (positions inside the sequence, row counts
// within the capacity, ids inside the vocabulary, k <= 8); a failed check
// aborts the kernel with the failed condition printed.  Release builds
// compile the checks away.
#ifdef SSM_DEBUG
#include <assert.h>
#define SSM_DCHECK(c) assert(c)
#else
#define SSM_DCHECK(c) ((void)0)
#endif
