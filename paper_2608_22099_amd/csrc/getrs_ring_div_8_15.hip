// Chain of column steps in the dividing forward mode (a lower triangular band
// with its diagonal), instantiated for K in [512, 1023] (one file per range keeps
// compiles parallel).
#include "getrs_ring.hpp"

namespace bandlu {

RingLaunch ring_launcher_div_8_15(int q) { return ring_launcher<kRingFwdDiv, 8, 15>(q); }

}  // namespace bandlu
