// Diagonal-pivot banded LU (getrf_diag.hpp) instantiated for ku = 9..16 (one
// file per range keeps compiles parallel).
#include "getrf_diag.hpp"

namespace bandlu {

WinKernel diag_kernel_ku9_16(int KU) {
    static constexpr auto table = DiagRange<9, 16>::make(std::make_integer_sequence<int, 16 - 9 + 1>{});
    return (KU >= 9 && KU <= 16) ? table[KU - 9] : nullptr;
}

}  // namespace bandlu
