// Chains of column steps on one vector, for bands up to K = 1023: the passes
// of the band solve with the LU factors (xGBTRS: the "lu(A) \ B" that
// Listings 1 and 2 end with) and of the other substitutions built on them
// (Listing 1's triangular solves, the transposed solve, the Cholesky solve).
//
// One workgroup of four wavefronts per right-hand side, one launch per pass.
// Step j finishes position j and updates positions j+1..j+K with one fused
// multiply-add each, in the order of the unblocked algorithm, so the result is
// bitwise that of the reference loops.  The entries of step j are
// AB[cb0 + col*ldab + e*es], e = 0..K, with col = j (forward) or n-1-j
// (backward), so a step can read a column of the band (es = 1) or a row
// (es = ldab-1).  Three modes:
//   kRingFwdLU  forward, unit diagonal, the row interchanges of ipiv first
//               (L of the LU factors: entry 0 is the diagonal, e the row j+e);
//   kRingBwd    positions reversed (position q is row n-1-q), x_j = b_j / entry K,
//               entry K-d updates the row d above (U with kv superdiagonals);
//   kRingFwdDiv forward, x_j = b_j / entry 0, no interchanges (a lower
//               triangular matrix with its diagonal).
//
// Wave 0 holds the right-hand side window in registers: slot s of lane L is
// position 64(B+s)+L while the steps of block B = j/64 run, C = Q+2 slots for
// K in [64Q, 64Q+63].  Finished slot 0 is stored at the end of the block and
// the slots move down by one; the slot that enters was loaded a block ahead.
// Per step the lane of position j is a compile-time constant (the step loop
// is unrolled by 64), so x_j reaches every lane by readlane, slot 0 takes the
// update above lane j, slots 1..Q-1 take it whole, and only slots Q and Q+1
// need a lane mask that depends on K: lanes <= j mod 64 + K - 64Q (- 64).
// Both masks come from one 128-bit register shifted by one each step.
//
// Waves 1..3 copy the factor columns of the next NB steps into one half of a
// double buffer in LDS while wave 0 works on the other half; one workgroup
// barrier per NB steps hands the halves over.  Column j's entries sit LDC
// apart in natural band order, so the value wave 0 needs for lane L, slot s
// is at a compile-time offset from one per-step address.
#pragma once

#include <utility>

#include "bufio.hpp"
#include "common.hpp"

namespace bandlu {

constexpr int kRingThreads = 256;  // wave 0 computes, waves 1..3 stage columns
constexpr int kLoaders = kRingThreads - 64;
constexpr int kPadLo = 128;        // LDS doubles before the buffers
constexpr int kPadHi = 128;        // and after
constexpr int kMaxQ = 15;          // K <= 1023

enum { kRingFwdLU = 0, kRingBwd = 1, kRingFwdDiv = 2 };

struct RingParams {
    const double *AB;
    const int32_t *ipiv;
    double *B;
    int64_t ldab, strideAB, strideP, ldb, strideB;
    int64_t cb0, es;    // entry e of step j at cb0 + col*ldab + e*es
    int n, kl, nrhs;    // kl: interchange reach (kRingFwdLU)
    int K, nsteps;      // positions a step updates; steps in the pass
};

// steps per LDS half-buffer: both halves of LDC = 64(Q+1) doubles per column
// stay below 150 KiB
template <int Q>
constexpr int ring_nb() { return Q <= 3 ? 32 : (Q <= 8 ? 16 : 8); }

template <int Q>
constexpr int ring_lds_doubles() { return kPadLo + 2 * ring_nb<Q>() * 64 * (Q + 1) + kPadHi; }

// lanes 0..x (x < 0: none, x >= 63: all)
__device__ __forceinline__ unsigned long long lanes_le(int x) {
    if (x < 0) return 0ull;
    if (x >= 63) return ~0ull;
    return (2ull << x) - 1ull;
}

__device__ __forceinline__ bool in_lanes(unsigned long long m) {
    return __builtin_amdgcn_inverse_ballot_w64(m);
}

template <int Q, int MODE>
__global__ __launch_bounds__(kRingThreads) void getrs_ring_kernel(RingParams P) {
    constexpr bool BWD = MODE == kRingBwd;
    constexpr int C = Q + 2;               // register slots of the window
    constexpr int NB = ring_nb<Q>();       // steps per LDS half-buffer
    constexpr int LDC = 64 * (Q + 1);      // LDS stride between columns (>= K + 1)
    constexpr int HALF = NB * LDC;
    __shared__ double lds[ring_lds_doubles<Q>()];

    const int tid = threadIdx.x;
    const int64_t sys = blockIdx.x;
    const int64_t bidx = sys / P.nrhs, krhs = sys - bidx * P.nrhs;
    const int n = P.n, ldab = int(P.ldab);
    const int K = P.K;
    const int nsteps = P.nsteps;
    const int nblk = (nsteps + NB - 1) / NB;
    const Buf ab = make_buf(P.AB + bidx * P.strideAB, uint32_t(int64_t(ldab) * n * 8));

    if (tid >= 64) {
        // ---------------------------------------------------- column staging --
        // Entries of step j: col = j forward, n-1-j backward; entry e at
        // cb0 + col*ldab + e*es (outside the band: read as zero, never used)
        constexpr int E = (LDC + kLoaders - 1) / kLoaders;  // entries per thread per column
        const int lt = tid - 64;
        // (every offset inside the band fits 32 bits: the band is below 2 GiB;
        // one unsigned compare rejects both ends)
        const uint32_t band = uint32_t(ldab) * uint32_t(n);
        const int esi = int(P.es), cb0 = int(P.cb0);
        const int lt_es = lt * esi, step_es = kLoaders * esi;
        // (a step's entries are consecutive in the common case es = 1, where
        // every one of them lies inside the band: that case keeps constant
        // offsets and no range check)
        const bool unit = esi == 1;
        auto stage = [&](int k) {
            double v[NB][E];
            if (unit) {
#pragma unroll
                for (int c = 0; c < NB; ++c) {
                    const int j = k * NB + c;
                    const int col = BWD ? n - 1 - j : j;
                    const int o0 = cb0 + col * ldab + lt;
#pragma unroll
                    for (int i = 0; i < E; ++i) {
                        const int e = lt + kLoaders * i;
                        const bool ok = j < nsteps && e <= K;
                        v[c][i] = buf_ld(ab, ok ? uint32_t(o0 + kLoaders * i) * 8u : kOutside);
                    }
                }
            } else {
#pragma unroll
                for (int c = 0; c < NB; ++c) {
                    const int j = k * NB + c;
                    const int col = BWD ? n - 1 - j : j;
                    const int o0 = cb0 + col * ldab + lt_es;
#pragma unroll
                    for (int i = 0; i < E; ++i) {
                        const int e = lt + kLoaders * i;
                        const uint32_t off = uint32_t(o0 + i * step_es);
                        const bool ok = j < nsteps && e <= K && off < band;
                        v[c][i] = buf_ld(ab, ok ? off * 8u : kOutside);
                    }
                }
            }
            double *dst = lds + kPadLo + (k & 1) * HALF;
#pragma unroll
            for (int c = 0; c < NB; ++c)
#pragma unroll
                for (int i = 0; i < E; ++i) {
                    const int e = lt + kLoaders * i;
                    if (e < LDC) dst[c * LDC + e] = v[c][i];
                }
        };
        if (nblk > 0) stage(0);
        for (int k = 0; k < nblk; ++k) {
            __syncthreads();  // block k staged; the half of block k-1 is free
            if (k + 1 < nblk) stage(k + 1);
        }
        return;
    }

    // --------------------------------------------------------- wave 0 --
    const int L = tid;
    const Buf xb = make_buf(P.B + bidx * P.strideB + krhs * P.ldb, uint32_t(int64_t(n) * 8));
    const Buf pb = make_buf(P.ipiv + bidx * P.strideP, uint32_t(int64_t(n) * 4));
    // position q <-> row (reversed in the backward pass)
    auto xoff = [&](int q) -> uint32_t {
        return (q >= 0 && q < n) ? uint32_t(BWD ? n - 1 - q : q) * 8u : kOutside;
    };
    double b[C];
#pragma unroll
    for (int s = 0; s < C; ++s) b[s] = buf_ld(xb, xoff(64 * s + L));
    double nxt = buf_ld(xb, xoff(64 * C + L));
    int ipv = 0, ipv_next = 0;
    if constexpr (MODE == kRingFwdLU) {
        ipv = buf_ld_i32(pb, L < n ? uint32_t(L) * 4u : kOutside);
        ipv_next = buf_ld_i32(pb, 64 + L < n ? uint32_t(64 + L) * 4u : kOutside);
    }
    const int r = K - 64 * Q;  // 0..63
    // slot Q takes lanes <= u + r, slot Q+1 lanes <= u + r - 64 (at u = 0: none)
    const unsigned long long mq0 = lanes_le(r);
    unsigned long long mq = mq0, mq1 = 0ull;
    // lanes > u at step u of a block: kept in scalar registers and shifted once
    // per step (opaque to constant folding, so no per-step constants are kept)
    unsigned long long above = ~1ull, onehot = 1ull;
    asm volatile("" : "+s"(above), "+s"(onehot));
    // per-lane LDS byte address of this lane's entry for slot C-1 (backward) or
    // slot 0 (forward) at the start of a half-buffer, before the step's offset
    // forward:  column base + 64 s + L - u
    // backward: column base + K - (64 s + L - u)
    const int lane_part = BWD ? (kPadLo + K - 64 * (C - 1) - L) : (kPadLo - 64 + L);
    int k = 0;           // LDS blocks entered
    bool live = nsteps > 0;
    double m[C];         // the step's factor entries by slot
    double dg = 0.0;     // dividing modes: the diagonal entry of the step
    uint32_t vhalf = 0;  // byte address of this lane's part in the current half

    auto fetch = [&]<int U>() __attribute__((always_inline)) {
        constexpr int c = U % NB;
#pragma unroll
        for (int s = 0; s < C; ++s) {
            // forward  index: base + c*LDC + 64 s + L - U  = (lane_part + 64) + c*LDC + 64 s - U
            // backward index: base + c*LDC + K - 64 s - L + U = lane_part + c*LDC + 64 (C-1-s) + U
            const int off = BWD ? (c * LDC + 64 * (C - 1 - s) + U) : (c * LDC + 64 + 64 * s - U);
            m[s] = *reinterpret_cast<const double *>(reinterpret_cast<const char *>(lds) + vhalf + off * 8);
        }
        if constexpr (MODE == kRingBwd) {
            // the diagonal entry e = K of the column (uniform address)
            dg = lds[kPadLo + (((k - 1) & 1) * HALF) + c * LDC + K];
        } else if constexpr (MODE == kRingFwdDiv) {
            dg = lds[kPadLo + (((k - 1) & 1) * HALF) + c * LDC];
        }
    };

    for (int B0 = 0; nsteps > 0; B0 += 64) {
        [&]<int... Us>(std::integer_sequence<int, Us...>) {
            (
                [&] {
                    constexpr int u = Us;
                    if (!live) return;
                    const int j = B0 + u;
                    if (j >= nsteps) {
                        live = false;
                        return;
                    }
                    if constexpr (u % NB == 0) {
                        __syncthreads();  // this half is staged
                        ++k;
                        vhalf = uint32_t(lane_part + ((k - 1) & 1) * HALF) * 8u;
                        fetch.template operator()<u>();
                    }
                    double xj;
                    if constexpr (MODE != kRingFwdLU) {
                        const double z = b[0] / dg;
                        xj = readlane_d(z, u);
                        if (in_lanes(onehot)) b[0] = xj;
                    } else {
                        int p = __builtin_amdgcn_readlane(ipv, u) - 1;
                        if (p != j) {
                            // exchange positions j and p (j < p <= j + kl): a row
                            // interchange of the forward pass
                            if (p > j && p <= j + P.kl && p < n) {
                                const int q = u + (p - j), sp = q >> 6, lp = q & 63;
                                const double vj = readlane_d(b[0], u);
                                double vp = 0.0;
#pragma unroll
                                for (int s = 0; s < C; ++s)
                                    if (s == sp) vp = readlane_d(b[s], lp);
#pragma unroll
                                for (int s = 0; s < C; ++s)
                                    if (s == sp && in_lanes(1ull << lp)) b[s] = vj;
                                if (in_lanes(onehot)) b[0] = vp;
                            }
                        }
                        xj = readlane_d(b[0], u);
                    }
                    double ms[C];
#pragma unroll
                    for (int s = 0; s < C; ++s) ms[s] = m[s];
                    // entries of the next step (same half-buffer)
                    if constexpr ((u + 1) % NB != 0 && u + 1 < 64) fetch.template operator()<u + 1>();
                    // ---- update positions j+1 .. j+K
                    {
                        // slot 0: lanes above u (a running mask, shifted once per step)
                        const unsigned long long m0mask = Q == 0 ? (above & mq) : above;
                        if (in_lanes(m0mask)) b[0] = __builtin_fma(-ms[0], xj, b[0]);
#pragma unroll
                        for (int s = 1; s < Q; ++s) b[s] = __builtin_fma(-ms[s], xj, b[s]);
                        if constexpr (Q >= 1) {
                            if (in_lanes(mq)) b[Q] = __builtin_fma(-ms[Q], xj, b[Q]);
                        }
                        if (in_lanes(mq1)) b[Q + 1] = __builtin_fma(-ms[Q + 1], xj, b[Q + 1]);
                        const unsigned long long carry = mq >> 63;
                        mq = (mq << 1) | 1ull;
                        mq1 = (mq1 << 1) | carry;
                        above <<= 1;
                        onehot <<= 1;
                    }
                    if constexpr (u == 63) {
                        // positions B0 .. B0+63 are final: store them, move the
                        // slots down, take the next block
                        buf_st(xb, xoff(B0 + L), b[0]);
#pragma unroll
                        for (int s = 0; s + 1 < C; ++s) b[s] = b[s + 1];
                        b[C - 1] = nxt;
                        nxt = buf_ld(xb, xoff(B0 + 64 * (C + 1) + L));
                        if constexpr (MODE == kRingFwdLU) {
                            ipv = ipv_next;
                            const int pi = B0 + 128 + L;
                            ipv_next = buf_ld_i32(pb, pi < n ? uint32_t(pi) * 4u : kOutside);
                        }
                        mq = mq0;
                        mq1 = 0ull;
                        above = ~1ull;
                        onehot = 1ull;
                        asm volatile("" : "+s"(above), "+s"(onehot));
                    }
                }(),
                ...);
        }(std::make_integer_sequence<int, 64>{});
        if (!live) {
            // the pass ended inside this block: every position held is final
#pragma unroll
            for (int s = 0; s < C; ++s) buf_st(xb, xoff(B0 + 64 * s + L), b[s]);
            break;
        }
    }
}


typedef void (*RingLaunch)(const RingParams &P, int64_t systems, hipStream_t s);

template <int Q, int MODE>
void ring_launch(const RingParams &P, int64_t systems, hipStream_t s) {
    hipLaunchKernelGGL((getrs_ring_kernel<Q, MODE>), dim3((unsigned)systems), dim3(kRingThreads), 0,
                       s, P);
}

// launchers of one pass for Q in [LO, HI] (one translation unit per range)
template <int MODE, int LO, int HI>
RingLaunch ring_launcher(int q) {
    RingLaunch f = nullptr;
    [&]<int... Is>(std::integer_sequence<int, Is...>) {
        ((q == LO + Is ? (f = &ring_launch<LO + Is, MODE>, 0) : 0), ...);
    }(std::make_integer_sequence<int, HI - LO + 1>{});
    return f;
}

RingLaunch ring_launcher_fwd_0_7(int q);
RingLaunch ring_launcher_fwd_8_15(int q);
RingLaunch ring_launcher_bwd_0_7(int q);
RingLaunch ring_launcher_bwd_8_15(int q);
RingLaunch ring_launcher_div_0_7(int q);
RingLaunch ring_launcher_div_8_15(int q);

// one pass of the chain for any K <= 1023 (the launcher for K's register group)
inline RingLaunch ring_pass(int mode, int K) {
    const int q = K >> 6;
    if (mode == kRingFwdLU) return q < 8 ? ring_launcher_fwd_0_7(q) : ring_launcher_fwd_8_15(q);
    if (mode == kRingBwd) return q < 8 ? ring_launcher_bwd_0_7(q) : ring_launcher_bwd_8_15(q);
    return q < 8 ? ring_launcher_div_0_7(q) : ring_launcher_div_8_15(q);
}

}  // namespace bandlu
