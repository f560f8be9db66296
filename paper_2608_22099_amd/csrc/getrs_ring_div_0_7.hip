// Chain of column steps in the dividing forward mode (a lower triangular band
// with its diagonal), instantiated for K in [0, 511] (one file per range keeps
// compiles parallel).
#include "getrs_ring.hpp"

namespace bandlu {

RingLaunch ring_launcher_div_0_7(int q) { return ring_launcher<kRingFwdDiv, 0, 7>(q); }

}  // namespace bandlu
