// The one-launch dataflow schedule of a search: the kernel k_flow (the
// protocol is described with FlowArgs in kernels.h) and its launch.
#include <hip/hip_ext.h>

#include "kernels.h"

namespace pase {

// Merge buffer of the row fills, one per workgroup.  The fills are calls of
// their own (below), so the buffer lives at file scope.
__shared__ MergeBuf<double> flow_xch_f64;
__shared__ MergeBuf<uint64_t> flow_xch_u64;

template <typename KeyT>
__device__ __forceinline__ MergeBuf<KeyT> &flow_xch();
template <>
__device__ __forceinline__ MergeBuf<double> &flow_xch<double>() { return flow_xch_f64; }
template <>
__device__ __forceinline__ MergeBuf<uint64_t> &flow_xch<uint64_t>() { return flow_xch_u64; }

// Descriptors are never written while the launch runs.  A wave-uniform
// pointer (call arguments and values read by one thread arrive in VGPRs) is
// moved to SGPRs and read through the constant address space, so that the
// descriptor -- and every address derived from it -- is read through the
// scalar unit, as a kernel reads its launch arguments.
// (readfirstlane works on signed 32-bit ints: each half is taken back to
// uint32_t before it is widened, or the low half would be sign-extended.)
template <typename T>
__device__ __forceinline__ const T &uniform_const(const T *p) {
    const uint64_t x = (uint64_t)(uintptr_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(x >> 32));
    const uint64_t u = ((uint64_t)hi << 32) | lo;
    return *(const T *)(const __attribute__((address_space(4))) T *)u;
}

// Every fill variant is a call of its own, so that its registers are
// allocated for it alone: inlined into one kernel, all variants share one
// allocation, sized for the worst point of any of them, and spill.
template <typename KeyT, int TZ, int TM, int NA>
__device__ __noinline__ void flow_rows_call(const RowsArgs *a, uint32_t b) {
    rows_item<KeyT, TZ, TM, NA>(uniform_const(a), __builtin_amdgcn_readfirstlane(b), flow_xch<KeyT>());
}

template <typename KeyT, int NT>
__device__ __noinline__ void flow_generic_call(const GenericArgs *a, uint32_t b) {
    generic_item<KeyT, NT>(uniform_const(a), __builtin_amdgcn_readfirstlane(b));
}

// An item the kernel cannot run (a variant it does not carry; the host never
// plans one for this launch) marks the search as failed instead of running.
__device__ __forceinline__ void flow_bad_variant(FlowCtl *ctl) {
    if (threadIdx.x == 0) __hip_atomic_store(&ctl->error, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename KeyT, int TZ, int TM, int NA>
__device__ __forceinline__ void flow_rows_v(const RowsArgs *a, uint32_t b, FlowCtl *ctl) {
    constexpr bool u64 = std::is_same<KeyT, uint64_t>::value;
    if constexpr (flow_rows_ok(u64, TZ, TM, NA < 0 ? 7 : NA)) flow_rows_call<KeyT, TZ, TM, NA>(a, b);
    else flow_bad_variant(ctl);
}

template <typename KeyT, int TZ, int TM>
__device__ __forceinline__ void flow_rows_tz(const RowsArgs *a, uint32_t na, uint32_t b, FlowCtl *ctl) {
    if constexpr (std::is_same<KeyT, double>::value) {
        switch (na) {
        case 0: flow_rows_v<KeyT, TZ, TM, 0>(a, b, ctl); break;
        case 1: flow_rows_v<KeyT, TZ, TM, 1>(a, b, ctl); break;
        case 2: flow_rows_v<KeyT, TZ, TM, 2>(a, b, ctl); break;
        case 3: flow_rows_v<KeyT, TZ, TM, 3>(a, b, ctl); break;
        default: flow_rows_v<KeyT, TZ, TM, 4>(a, b, ctl); break;
        }
    } else {
        flow_rows_v<KeyT, TZ, TM, -1>(a, b, ctl);
    }
}

// variant = (TZ * 4 + TM) * 8 + NA, the encoding of the batched launches
template <typename KeyT>
__device__ __forceinline__ void flow_rows(const RowsArgs *a, uint32_t variant, uint32_t b, FlowCtl *ctl) {
    const uint32_t na = variant % 8;
    switch (variant / 8) {
    case 1 * 4 + 1: flow_rows_tz<KeyT, 1, 1>(a, na, b, ctl); break;
    case 1 * 4 + 2: flow_rows_tz<KeyT, 1, 2>(a, na, b, ctl); break;
    case 8 * 4 + 1: flow_rows_tz<KeyT, 8, 1>(a, na, b, ctl); break;
    case 8 * 4 + 2: flow_rows_tz<KeyT, 8, 2>(a, na, b, ctl); break;
    case 12 * 4 + 1: flow_rows_tz<KeyT, 12, 1>(a, na, b, ctl); break;
    case 12 * 4 + 2: flow_rows_tz<KeyT, 12, 2>(a, na, b, ctl); break;
    case 14 * 4 + 1: flow_rows_tz<KeyT, 14, 1>(a, na, b, ctl); break;
    case 14 * 4 + 2: flow_rows_tz<KeyT, 14, 2>(a, na, b, ctl); break;
    case 16 * 4 + 1: flow_rows_tz<KeyT, 16, 1>(a, na, b, ctl); break;
    case 16 * 4 + 2: flow_rows_tz<KeyT, 16, 2>(a, na, b, ctl); break;
    case 24 * 4 + 1: flow_rows_tz<KeyT, 24, 1>(a, na, b, ctl); break;
    case 28 * 4 + 1: flow_rows_tz<KeyT, 28, 1>(a, na, b, ctl); break;
    default: flow_bad_variant(ctl); break;
    }
}

template <typename KeyT>
__device__ __forceinline__ void flow_generic(const GenericArgs *a, uint32_t variant, uint32_t b) {
    switch (variant) {
    case 1: flow_generic_call<KeyT, 1>(a, b); break;
    case 2: flow_generic_call<KeyT, 2>(a, b); break;
    case 3: flow_generic_call<KeyT, 3>(a, b); break;
    case 4: flow_generic_call<KeyT, 4>(a, b); break;
    case 5: flow_generic_call<KeyT, 5>(a, b); break;
    case 6: flow_generic_call<KeyT, 6>(a, b); break;
    default: flow_generic_call<KeyT, -1>(a, b); break;
    }
}

template <typename KeyT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) void k_flow(FlowArgs f) {
    __shared__ uint32_t s_q, s_t;
    constexpr uint32_t kNone = 2;
    bool lat = blockIdx.x < f.lat_workers;   // thread 0's role
    for (;;) {
        if (threadIdx.x == 0) {
            uint32_t q = kNone, t = 0;
            if (lat) {
                t = atomicAdd(&f.ctl->head[kLatQ], 1u);
                if (t < f.nitems[kLatQ]) q = kLatQ;
                else lat = false;
            }
            if (q == kNone) {
                const uint32_t h = load_counter(&f.ctl->head[kLatQ]);
                if (h < f.nitems[kLatQ]) {
                    const Seg &sg = f.seg[kLatQ][seg_find(f.seg[kLatQ], f.nseg[kLatQ], h)];
                    if (deps_met(f, sg) && atomicCAS(&f.ctl->head[kLatQ], h, h + 1) == h) {
                        q = kLatQ;
                        t = h;
                    }
                }
            }
            if (q == kNone) {
                t = atomicAdd(&f.ctl->head[kBulkQ], 1u);
                if (t < f.nitems[kBulkQ]) {
                    q = kBulkQ;
                } else {
                    t = atomicAdd(&f.ctl->head[kLatQ], 1u);
                    if (t < f.nitems[kLatQ]) q = kLatQ;
                }
            }
            s_q = q;
            s_t = t;
        }
        __syncthreads();
        const uint32_t q = __builtin_amdgcn_readfirstlane(s_q), t = __builtin_amdgcn_readfirstlane(s_t);
        if (q == kNone) break;   // uniform: both queues are drained
        const Seg &sg = uniform_const(&f.seg[q][seg_find(f.seg[q], f.nseg[q], t)]);
        if (threadIdx.x == 0 && !deps_met(f, sg)) {
            const uint64_t t0 = wall_clock64();
            for (uint32_t k = sg.dep_begin; k < sg.dep_end; k++) {
                const SegDep d = f.deps[k];
                while (load_counter(&f.done[d.counter]) < d.target) {
                    if (load_counter(&f.ctl->error)) break;
                    if (wall_clock64() - t0 > f.timeout_ticks) {
                        __hip_atomic_store(&f.ctl->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(2);
                }
            }
        }
        __syncthreads();
        // every wave: drop stale cached copies of what other workgroups published
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const uint32_t b = t - sg.first;
        if (b >= sg.count) {   // (the host builds the queues so that this cannot happen)
            flow_bad_variant(f.ctl);
        } else switch (sg.kind) {
        case kSegPrep: prep_item<KeyT>(uniform_const(&f.prep[sg.pos]), b, f.V, f.E, f.L, f.lsum, f.sig, f.cb, f.r); break;
        case kSegRows: flow_rows<KeyT>(&f.rows[sg.pos], sg.variant, b, f.ctl); break;
        case kSegGeneric: flow_generic<KeyT>(&f.gen[sg.pos], sg.variant, b); break;
        default: reduce_item<KeyT>(uniform_const(&f.red[sg.pos]), b); break;
        }
        // publish: every thread's stores become visible at device scope, then
        // the item is counted (the barrier also retires this round's s_q/s_t)
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) __hip_atomic_fetch_add(&f.done[sg.pos], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <typename KeyT>
hipError_t flow_occupancy(int *per_cu) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, k_flow<KeyT>, 256, 0);
}

template <typename KeyT>
hipError_t flow_launch(const FlowArgs &f, uint32_t grid, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL((k_flow<KeyT>), dim3(grid), dim3(256), 0, s, e0, e1, 0, f);
    return hipGetLastError();
}

template hipError_t flow_occupancy<double>(int *);
template hipError_t flow_occupancy<uint64_t>(int *);
template hipError_t flow_launch<double>(const FlowArgs &, uint32_t, hipStream_t, hipEvent_t, hipEvent_t);
template hipError_t flow_launch<uint64_t>(const FlowArgs &, uint32_t, hipStream_t, hipEvent_t, hipEvent_t);

}  // namespace pase
