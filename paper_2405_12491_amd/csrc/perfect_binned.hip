// perfect_binned.hip -- the generic PERFECT kernel on tiles of 16- or 8-bit feature bins.
#include "perfect_kernel.h"

namespace bridger {

template <int D>
static int launch_binned_d(const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                           void *stream) {
  if (a.x_bytes == 2) return launch_perfect_dfx<D, true, 2>(a, waves, n_wg, lds_bytes, stream);
  if (a.x_bytes == 1) return launch_perfect_dfx<D, true, 1>(a, waves, n_wg, lds_bytes, stream);
  return (int)hipErrorInvalidValue;
}

int launch_perfect_binned(int depth, const LaunchArgs &a, int waves, int64_t n_wg, int lds_bytes,
                          void *stream) {
  switch (depth) {
    case 1: return launch_binned_d<1>(a, waves, n_wg, lds_bytes, stream);
    case 2: return launch_binned_d<2>(a, waves, n_wg, lds_bytes, stream);
    case 3: return launch_binned_d<3>(a, waves, n_wg, lds_bytes, stream);
    case 4: return launch_binned_d<4>(a, waves, n_wg, lds_bytes, stream);
    case 5: return launch_binned_d<5>(a, waves, n_wg, lds_bytes, stream);
    case 6: return launch_binned_d<6>(a, waves, n_wg, lds_bytes, stream);
    case 7: return launch_binned_d<7>(a, waves, n_wg, lds_bytes, stream);
    case 8: return launch_binned_d<8>(a, waves, n_wg, lds_bytes, stream);
    case 9: return launch_binned_d<9>(a, waves, n_wg, lds_bytes, stream);
    case 10: return launch_binned_d<10>(a, waves, n_wg, lds_bytes, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

}  // namespace bridger
