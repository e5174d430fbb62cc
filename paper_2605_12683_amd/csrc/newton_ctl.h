// Pass-end control of the adaptive Newton loop on the device, shared by the kernels that take
// it themselves (internal to libdeer, not part of the ABI).
#pragma once

#include "common.h"
#include "launch.h"

namespace deer {

// Convergence test and update safeguard of one pass for sequence b from its maxima e = max
// |Delta| bits and zm = max |z| bits: accept the update (flip sel, count it, relax the damping,
// freeze the sequence once max|Delta| < tol), or reject it (keep sel, raise the damping:
// 1 - gamma = first, then x grow up to 1 = the fixed-point step); a non-finite fixed-point step
// ends the sequence.
// tag: with nd.pv, the number of the pass that may use the aggregates the caller's kernel
// formed for the accepted iterate (it is stored when the update is kept and the sequence goes on)
__device__ __forceinline__ void seq_decide(int b, uint32_t e, uint32_t zm, const NewtonDev &nd, float tol, float bound,
                                           const NewtonDamp &dp, uint32_t tag = 0u) {
    const float ef = __uint_as_float(e), zf = __uint_as_float(zm);
    const bool fin = e < 0x7f800000u;
    float om = nd.om[b];
    const bool keep = fin && (bound < 0.f || om >= 1.f || ef <= bound * (1.f + zf));
    // a stopped sequence: device control block, then the host block (act last)
    auto stop = [&](int it, int status) {
        nd.act[b] = 0;
        nd.status[b] = status;
        if (nd.hact) {
            nd.hit[b] = it;
            nd.hnorm[b] = ef;
            nd.hstat[b] = status;
            __hip_atomic_store(nd.hact + b, 0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    };
    if (keep) {
        nd.sel[b] ^= 1;
        const int it = nd.it[b] + 1;
        nd.it[b] = it;
        nd.norm[b] = ef;
        if (om > 0.f) om = om / dp.shrink < dp.floor ? 0.f : om / dp.shrink;
        if (ef < tol) stop(it, 1);
        else if (nd.pv) nd.pv[b] = tag;
    } else if (om >= 1.f) {
        nd.norm[b] = ef;
        stop(nd.it[b], 2);
    } else {
        om = om == 0.f ? dp.first : fminf(1.f, om * dp.grow);
    }
    nd.om[b] = om;
    nd.gamma[b] = 1.f - om;
}

// Arrival of `cnt` chains of sequence b with maxima e, zm (see FusedCtl).  Device-scope atomics
// meet at one coherence point across the XCDs; each maximum is returned (so performed) before
// the count is raised, so the chain that completes the count reads the final maxima.
__device__ __forceinline__ void seq_arrive(const FusedCtl &fc, int b, int cnt, int ncs, uint32_t e, uint32_t zm,
                                           uint32_t tag = 0u) {
    uint32_t *blk = fc.seq + (size_t)b * kSeqWords;   // count | max |Delta| | max |z|, 128 bytes apart
    const uint32_t r1 = __hip_atomic_fetch_max(blk + 32, e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t r2 = __hip_atomic_fetch_max(blk + 64, zm, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the count may only move once both maxima are in: the increment depends on their return
    // values (|x| bits are below 2^31, so the added term is zero)
    const uint32_t old = __hip_atomic_fetch_add(blk, (uint32_t)cnt + ((r1 | r2) >> 31), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    if (old + (uint32_t)cnt != (uint32_t)ncs) return;
    const uint32_t ef = __hip_atomic_load(blk + 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t zf = __hip_atomic_load(blk + 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    seq_decide(b, ef, zf, fc.nd, fc.tol, fc.bound, fc.dp, tag);
    __hip_atomic_store(blk + 32, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(blk + 64, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(blk, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace deer
