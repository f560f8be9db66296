// Ring-window band solve, forward (L and interchanges) pass, instantiated for
// kl in [0, 511] (one file per range keeps compiles parallel).
#include "getrs_ring.hpp"

namespace bandlu {

RingLaunch ring_launcher_fwd_0_7(int q) { return ring_launcher<kRingFwdLU, 0, 7>(q); }

}  // namespace bandlu
