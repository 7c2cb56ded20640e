// Host-side access to the RoPE angle reduction of the device helpers, so a CPU
// test can compare it with an exact reduction.  Built by tests/test_rope_reduce.py.
#include "../paper_2608_30252_amd/csrc/mad_device.h"

extern "C" void rope_reduce_many(const double *a, double *r, int n) {
    for (int i = 0; i < n; ++i) r[i] = mad::rope_reduce(a[i]);
}
