// Ring-window band solve, backward (U) pass, instantiated for
// kl+ku in [512, 1023] (one file per range keeps compiles parallel).
#include "getrs_ring.hpp"

namespace bandlu {

RingLaunch ring_launcher_bwd_8_15(int q) { return ring_launcher<kRingBwd, 8, 15>(q); }

}  // namespace bandlu
