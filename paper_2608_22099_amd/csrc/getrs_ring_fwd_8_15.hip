// Ring-window band solve, forward (L and interchanges) pass, instantiated for
// kl in [512, 1023] (one file per range keeps compiles parallel).
#include "getrs_ring.hpp"

namespace bandlu {

RingLaunch ring_launcher_fwd_8_15(int q) { return ring_launcher<kRingFwdLU, 8, 15>(q); }

}  // namespace bandlu
