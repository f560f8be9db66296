// Ring-window band solve, backward (U) pass, instantiated for
// kl+ku in [0, 511] (one file per range keeps compiles parallel).
#include "getrs_ring.hpp"

namespace bandlu {

RingLaunch ring_launcher_bwd_0_7(int q) { return ring_launcher<kRingBwd, 0, 7>(q); }

}  // namespace bandlu
