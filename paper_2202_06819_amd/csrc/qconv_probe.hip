// Measurement aids: a kernel that issues nothing but int8 MFMAs, so the rate
// the matrix cores sustain on this device (and the shader clock they ran at)
// can be measured beside the convolution kernels; and an empty kernel, whose
// time per launch is the fixed cost every launch of a grid pays.  Neither
// computes anything of the convolution.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "qconv_internal.h"

namespace qconv {

namespace {

typedef int v4i_p __attribute__((ext_vector_type(4)));

constexpr int kProbeChains = 8;   // independent accumulators per wave: covers the MFMA's dependent-issue latency

// Four waves per workgroup (one per SIMD when a CU holds one workgroup); each
// wave runs `iters` rounds of independent int8 MFMAs: eight chains of
// v_mfma_i32_16x16x64_i8 (WIDE = false) or four of v_mfma_i32_32x32x32_i8
// (WIDE = true) -- the same int8 operations per round either way.
// Wave 0 of every workgroup records the shader-clock counter and the 100 MHz
// constant counter around its loop.
typedef int v16i_p __attribute__((ext_vector_type(16)));
template <bool WIDE>
__global__ void __launch_bounds__(256) mfma_i8_probe(int iters, int32_t *sink, uint64_t *stamps) {
    const int tid = threadIdx.x;
    const v4i_p a = {tid, tid * 7 + 1, tid ^ 0x55, tid + 0x01010101};
    const v4i_p b = {tid * 3, tid + 5, ~tid, tid << 8};
    constexpr int kChains = WIDE ? kProbeChains / 2 : kProbeChains;
    typedef typename std::conditional<WIDE, v16i_p, v4i_p>::type Acc;
    Acc acc[kChains];
#pragma unroll
    for (int j = 0; j < kChains; ++j)
#pragma unroll
        for (int e = 0; e < (WIDE ? 16 : 4); ++e) acc[j][e] = tid + j + e;
    const uint64_t c0 = clock64();
    const uint64_t r0 = wall_clock64();
    for (int i = 0; i < iters; ++i) {
        // tied operands keep each accumulator in place (no copies between rounds)
#pragma unroll
        for (int j = 0; j < kChains; ++j) {
            if constexpr (WIDE)
                asm volatile("v_mfma_i32_32x32x32_i8 %0, %1, %2, %0" : "+v"(acc[j]) : "v"(a), "v"(b));
            else
                asm volatile("v_mfma_i32_16x16x64_i8 %0, %1, %2, %0" : "+v"(acc[j]) : "v"(a), "v"(b));
        }
    }
    // the accumulators are read by VALU below: let the last MFMAs retire first
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
    const uint64_t c1 = clock64();
    const uint64_t r1 = wall_clock64();
    int32_t s = 0;
#pragma unroll
    for (int j = 0; j < kChains; ++j)
#pragma unroll
        for (int e = 0; e < (WIDE ? 16 : 4); ++e) s += acc[j][e];
    sink[(size_t)blockIdx.x * 256 + tid] = s;
    if (tid == 0) {
        uint64_t *st = stamps + (size_t)blockIdx.x * 4;
        st[0] = c0;
        st[1] = c1;
        st[2] = r0;
        st[3] = r1;
    }
}

// Does nothing: its launches measure the cost of dispatching a grid of this
// shape (and dynamic LDS size) and of waiting for it to drain.
__global__ void __launch_bounds__(1024) empty_probe() {}

// One wave: the arrival counters of the meeting probe start each launch at 0
// (a kernel rather than a memset, so the pair can also sit in a graph).
__global__ void __launch_bounds__(64) zero_counters(uint32_t *arrivals) {
    if (threadIdx.x < kMeetCounters) __hip_atomic_store(arrivals + threadIdx.x * kMeetStride, 0u, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
}

// A grid that meets `rounds` times inside one launch.  At each meeting every
// workgroup makes its earlier writes visible to the whole device (agent-scope
// release), counts itself in, polls until the whole grid has arrived at this
// meeting, and acquires (agent scope) before it goes on -- what a network run
// as one persistent launch would pay at each layer boundary instead of a
// kernel launch.  Counting in: flat, one atomic add per workgroup on one
// counter; two-level, one add on its group's counter (workgroups are dealt to
// the eight XCDs round robin, so a group is the workgroups of one XCD) and the
// last of each group adds the group's arrival to the top counter.  The grid
// must be co-resident (the host allows at most one workgroup per CU).  The
// wait is bounded: after `spin_limit` polls a workgroup writes 1 to *err and
// leaves, so every workgroup ends even if some never arrive.
__global__ void __launch_bounds__(256) grid_meet_probe(int rounds, int two_level, int spin_limit, uint32_t *arrivals,
                                                       int32_t *err) {
    __shared__ int gave_up;
    const uint32_t ngroups = gridDim.x < 8 ? gridDim.x : 8u;
    const uint32_t grp = blockIdx.x & 7u;
    const uint32_t gsize = (gridDim.x - grp + 7u) / 8u;   // workgroups of this group
    for (int r = 0; r < rounds; ++r) {
        __syncthreads();
        if (threadIdx.x == 0) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            uint32_t target;
            if (two_level) {
                const uint32_t old = __hip_atomic_fetch_add(arrivals + (1u + grp) * kMeetStride, 1u, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                if (old == (uint32_t)(r + 1) * gsize - 1u)   // the group's last arrival
                    __hip_atomic_fetch_add(arrivals, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                target = (uint32_t)(r + 1) * ngroups;
            } else {
                __hip_atomic_fetch_add(arrivals, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                target = (uint32_t)(r + 1) * gridDim.x;
            }
            bool here = false;
            for (int polls = 0; polls < spin_limit; ++polls) {
                if (__hip_atomic_load(arrivals, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) {
                    here = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            if (!here) __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            gave_up = here ? 0 : 1;
        }
        __syncthreads();
        if (gave_up) return;   // uniform over the workgroup
    }
}

}  // namespace

hipError_t launch_empty_probe(int blocks, int threads, int lds_bytes, hipStream_t stream) {
    if (lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&empty_probe),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(empty_probe, dim3((unsigned)blocks), dim3((unsigned)threads), (size_t)lds_bytes, stream);
    return hipGetLastError();
}

hipError_t launch_meet_probe(int blocks, int rounds, int two_level, int spin_limit, uint32_t *arrivals, int32_t *err,
                             hipStream_t stream) {
    hipLaunchKernelGGL(zero_counters, dim3(1), dim3(64), 0, stream, arrivals);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(grid_meet_probe, dim3((unsigned)blocks), dim3(256), 0, stream, rounds, two_level, spin_limit,
                       arrivals, err);
    return hipGetLastError();
}

int64_t mfma_probe_ops(int blocks, int iters) {
    return (int64_t)blocks * 4 * iters * kProbeChains * (2 * 16 * 16 * 64);
}

hipError_t launch_mfma_probe(int blocks, int iters, bool wide, int32_t *sink, uint64_t *stamps, hipStream_t stream) {
    if (wide)
        hipLaunchKernelGGL(mfma_i8_probe<true>, dim3((unsigned)blocks), dim3(256), 0, stream, iters, sink, stamps);
    else
        hipLaunchKernelGGL(mfma_i8_probe<false>, dim3((unsigned)blocks), dim3(256), 0, stream, iters, sink, stamps);
    return hipGetLastError();
}

}  // namespace qconv
