// Cross-workgroup exchange and grid barrier of the persistent kernels
// (device side), shared by every persistent launch of the library.
#pragma once

#include <hip/hip_runtime.h>

#include "device.h"
#include "kernels.h"

namespace lsd {

// ---------------------------------------------------------------------------
// Cross-workgroup exchange and grid barrier.
//
// Values that other workgroups read during the same launch (the compacted
// h_t, x_t and gx_t of the forward stack, the backward DA_t and dx_t) are
// written with relaxed agent-scope atomic stores (ordinary stores carrying
// the device-coherence bit, written through to the coherent level), so a
// producer never writes back its L2, and read with device-coherent loads
// (16-byte buffer loads with the SC1 bit, the form of an agent-scope atomic
// load), so a consumer needs no cache invalidation.  A workgroup signals the
// end of a step by waiting for its own stores to complete, synchronising its
// threads and adding 1 to its slot's counter; a waiting workgroup spins (one
// wave) until the counter shows the step complete.  The spin is bounded by
// wall-clock time; on time-out, or when another workgroup has timed out, it
// reports failure and the kernel ends (outputs are then poisoned with NaN).
// A slot's counter is split over BAR_LINES cache lines (workgroup j adds to
// line j % BAR_LINES, lanes of the waiting wave poll one line each): the
// atomic adds of one line are serialised, and with one line per slot a step
// of 82 workgroups spent about 0.5 us more in the barrier.  Waits are on
// step counts: line k of slot d reaches s * (the number of the slot's
// workgroups on line k) once step s is complete.

// workgroups of slot `slot` (blocks [slot*nslot, (slot+1)*nslot)) that add
// to line i
__device__ __forceinline__ unsigned bar_count(int nslot, int slot, int i) {
    auto upto = [&](int n) { return n > i ? (n - i + BAR_LINES - 1) / BAR_LINES : 0; };
    return (unsigned)(upto((slot + 1) * nslot) - upto(slot * nslot));
}
__device__ __forceinline__ unsigned* slot_bar(unsigned* bar, int slot) { return bar + BAR_PITCH * BAR_LINES * slot; }
// the sticky status word of the step, beside the error flag
__device__ __forceinline__ int* sync_status(int* err) { return (int*)((char*)err + (SYNC_STATUS_OFS - SYNC_ERR_OFS)); }

__device__ __forceinline__ void grid_arrive(unsigned* sbar) {
    __builtin_amdgcn_s_waitcnt(0);      // this thread's stores have completed
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_fetch_add(sbar + BAR_PITCH * (blockIdx.x % BAR_LINES), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until slot `slot` (counter lines at sbar) has completed `steps`
// steps, and, with sbar2, slot `slot2` has completed `steps2` (lanes 0-15
// poll the first slot's lines, lanes 16-31 the second's, in the same loop:
// no extra round trip).  Returns false on time-out or when another workgroup
// has timed out (err set).  With seen / seen2 (LDS), also records the number
// of steps the lines read last show as complete.
__device__ __forceinline__ bool grid_wait(unsigned* sbar, int slot, int nslot, unsigned steps, int* err,
                                          long long timeout, int fail_bit, unsigned* seen = nullptr,
                                          unsigned* sbar2 = nullptr, int slot2 = 0, unsigned steps2 = 0,
                                          unsigned* seen2 = nullptr) {
    __shared__ int ok;
    if (timeout <= 0) {
        // a zero time-out (set from the host, for tests of the failure
        // path): every wait fails at once, so every workgroup leaves through
        // the time-out path without spinning.  The flags are set before the
        // workgroup barrier, so every thread reads them set afterwards.
        if (threadIdx.x == 0) {
            __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_or(sync_status(err), fail_bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __builtin_amdgcn_s_waitcnt(0);      // both have completed
        }
        __syncthreads();
        return false;
    }
    if (threadIdx.x < 64) {
        const int i = threadIdx.x;
        const bool second = i >= BAR_LINES;
        const int li = i & (BAR_LINES - 1);
        const unsigned n = i < BAR_LINES ? bar_count(nslot, slot, li)
                         : (i < 2 * BAR_LINES && sbar2) ? bar_count(nslot, slot2, li) : 0u;
        const unsigned* line = (second && sbar2 ? sbar2 : sbar) + BAR_PITCH * li;
        const unsigned want = (second ? steps2 : steps) * n;
        int good = 1;
        const long long t0 = wall_clock64();
        unsigned v = 0;
        // (the error flag is read only once a wait has taken a while: a load
        // of it in every poll made the barrier 0.2 us slower)
        for (;;) {
            v = n ? __hip_atomic_load(line, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
            if (__builtin_amdgcn_ballot_w64(n != 0 && v < want) == 0) break;
            const long long el = wall_clock64() - t0;
            if (el > timeout) {
                if (i == 0) {
                    __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_fetch_or(sync_status(err), fail_bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __builtin_amdgcn_s_waitcnt(0);
                }
                good = 0;
                break;
            }
            if (el > (timeout >> 12)) {
                const int e = i == 0 ? __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
                if (__builtin_amdgcn_ballot_w64(e != 0) != 0) { good = 0; break; }
            }
        }
        if (seen || seen2) {
            // steps complete per lane; the minimum over each half of the wave
            unsigned c = n ? v / n : 0xffffffffu;
#pragma unroll
            for (int o = BAR_LINES / 2; o; o >>= 1) c = min(c, (unsigned)__shfl_xor((int)c, o));
            if (seen && i == 0) *seen = c;
            if (seen2 && i == BAR_LINES) *seen2 = c;
        }
        if (i == 0) ok = good;
    }
    // every read of what other workgroups of this launch published is a
    // device-coherent load (SC1), issued after this point: no cache needs
    // invalidating (an agent-scope acquire would invalidate the XCD's L2 from
    // every workgroup, which cost up to 0.9 us per barrier at 123 workgroups)
    __syncthreads();
    return ok != 0;
}

// Every workgroup ends here, past its last barrier wait; the last one to
// arrive returns the step counters, the error flag and the exit counter to
// zero, so the next launch starts clear without a clearing kernel.  (The
// outputs' time-out check comes before: the flag is read by then.  A
// time-out stays recorded in the sticky status word, which this does not
// clear.)
__device__ __forceinline__ void grid_exit(unsigned* bar, int nslots, int* err) {
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned* ex = slot_bar(bar, BAR_EXIT);
        const unsigned tk = __hip_atomic_fetch_add(ex, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        if (tk == gridDim.x - 1) {
            for (int i = 0; i < nslots * BAR_LINES; ++i)
                __hip_atomic_store(bar + BAR_PITCH * i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(ex, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// coherent store of element i of a buffer of n elements: a buffer store with
// the device-coherence bit (as xstore) at a 32-bit offset
__device__ __forceinline__ void store_coherent(bf16* base, size_t n, uint32_t i, bf16 v) {
    __builtin_amdgcn_raw_buffer_store_b16(v, buf_rsrc(base, (uint32_t)(n * 2)), i * 2u, 0, CPOL_SC1);
}
__device__ __forceinline__ void store_coherent(float* base, size_t n, uint32_t i, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), buf_rsrc(base, (uint32_t)(n * 4)), i * 4u, 0, CPOL_SC1);
}

// coherent (agent-scope) element store and 8-element load of exchange data
__device__ __forceinline__ void xstore(bf16* p, bf16 v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void xstore(float* p, float v) {
    __hip_atomic_store((uint32_t*)p, __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void xload8(const bf16* p, bf16* o) {
    const unsigned long long* q = (const unsigned long long*)p;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const unsigned long long v = __hip_atomic_load(q + h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int e = 0; e < 4; ++e) o[4 * h + e] = (bf16)((v >> (16 * e)) & 0xffffu);
    }
}
__device__ __forceinline__ void xload8(const float* p, float* o) {
    const unsigned long long* q = (const unsigned long long*)p;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const unsigned long long v = __hip_atomic_load(q + h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        o[2 * h] = __uint_as_float((uint32_t)v);
        o[2 * h + 1] = __uint_as_float((uint32_t)(v >> 32));
    }
}

// coherent load of one float
__device__ __forceinline__ float xload1(const float* p) {
    return __uint_as_float(__hip_atomic_load((const uint32_t*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

// coherent load of 4 consecutive elements (8-byte aligned bf16 / 16-byte f32)
__device__ __forceinline__ void xload4(const bf16* p, bf16* o) {
    const unsigned long long v = __hip_atomic_load((const unsigned long long*)p, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = (bf16)((v >> (16 * e)) & 0xffffu);
}
__device__ __forceinline__ void xload4(const float* p, float* o) {
    const unsigned long long* q = (const unsigned long long*)p;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const unsigned long long v = __hip_atomic_load(q + h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        o[2 * h] = __uint_as_float((uint32_t)v);
        o[2 * h + 1] = __uint_as_float((uint32_t)(v >> 32));
    }
}
// 4 consecutive elements, plain load (8-byte aligned bf16 / 16-byte f32)
__device__ __forceinline__ void ld4g(const bf16* p, bf16* o) {
    const uint2 v = *(const uint2*)p;
    o[0] = (bf16)(v.x & 0xffffu); o[1] = (bf16)(v.x >> 16);
    o[2] = (bf16)(v.y & 0xffffu); o[3] = (bf16)(v.y >> 16);
}
__device__ __forceinline__ void ld4g(const float* p, float* o) {
    const float4 v = *(const float4*)p;
    o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
}
// 8 consecutive elements (LDS or global, 16-byte aligned)
__device__ __forceinline__ void lds8(const bf16* p, bf16* o) {
    const uint4 v = *(const uint4*)p;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (bf16)((w[e >> 1] >> (16 * (e & 1))) & 0xffffu);
}
__device__ __forceinline__ void lds8(const float* p, float* o) {
    const float4 v0 = *(const float4*)p, v1 = *(const float4*)(p + 4);
    o[0] = v0.x; o[1] = v0.y; o[2] = v0.z; o[3] = v0.w;
    o[4] = v1.x; o[5] = v1.y; o[6] = v1.z; o[7] = v1.w;
}


}  // namespace lsd
