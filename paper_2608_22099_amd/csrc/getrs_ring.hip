// Host side of the ring-window band solve (getrs_ring.hpp): variant check
// and the two launches (forward, backward) of one solve.
#include <algorithm>

#include "getrs_ring.hpp"

namespace bandlu {

int launch_getrs_ring(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                      double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s);
bool getrs_ring_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab);

bool getrs_ring_fits(int64_t n, int64_t kl, int64_t ku, int64_t ldab) {
    return (kl + ku) >> 6 <= kMaxQ && ldab * n * 8 <= kMaxBufferBytes && n * 8 <= kMaxBufferBytes;
}

int launch_getrs_ring(int64_t n, int64_t kl, int64_t ku, int64_t nrhs, const double *dAB,
                      int64_t ldab, int64_t strideAB, const int32_t *d_ipiv, int64_t strideP,
                      double *dB, int64_t ldb, int64_t strideB, int64_t batch, hipStream_t s) {
    if (n == 0 || nrhs == 0 || batch == 0) return BANDLU_OK;
    if (!getrs_ring_fits(n, kl, ku, ldab)) {
        set_error("band_getrs: the ring solve needs kl+ku <= %d and a band below 2 GiB",
                  64 * (kMaxQ + 1) - 1);
        return BANDLU_ERR_UNSUPPORTED;
    }
    RingParams P;
    P.AB = dAB;
    P.ipiv = d_ipiv;
    P.B = dB;
    P.ldab = ldab;
    P.strideAB = strideAB;
    P.strideP = strideP;
    P.ldb = ldb;
    P.strideB = strideB;
    P.n = (int)n;
    P.kl = (int)kl;
    P.nrhs = (int)nrhs;
    const int64_t systems = batch * nrhs;
    if (kl > 0 && n > 1) {
        // unit L with the interchanges: column j's entries from the diagonal row kv
        P.cb0 = kl + ku;
        P.es = 1;
        P.K = (int)kl;
        P.nsteps = (int)n - 1;
        ring_pass(kRingFwdLU, P.K)(P, systems, s);
        BANDLU_CHECK_LAUNCH("band_getrs (ring, forward)");
    }
    // U: column n-1-j's entries from row 0 (U(col-kv+e, col))
    P.cb0 = 0;
    P.es = 1;
    P.K = (int)(kl + ku);
    P.nsteps = (int)n;
    ring_pass(kRingBwd, P.K)(P, systems, s);
    BANDLU_CHECK_LAUNCH("band_getrs (ring, backward)");
    return BANDLU_OK;
}

}  // namespace bandlu
