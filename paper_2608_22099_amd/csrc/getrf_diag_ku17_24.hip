// Diagonal-pivot banded LU (getrf_diag.hpp) instantiated for ku = 17..24 (one
// file per range keeps compiles parallel).
#include "getrf_diag.hpp"

namespace bandlu {

WinKernel diag_kernel_ku17_24(int KU) {
    static constexpr auto table = DiagRange<17, 24>::make(std::make_integer_sequence<int, 24 - 17 + 1>{});
    return (KU >= 17 && KU <= 24) ? table[KU - 17] : nullptr;
}

}  // namespace bandlu
