// hc_aggregate.hip -- the aggregation step between the two phases of
// Algorithm 1, run on one GPU in place of the switch / AllReduce:
// Y <- sum over workers of Y_w, B <- OR over workers of B_w (section 3).
//
// A pure HBM stream: every lane reads one 16-byte vector (when the buffers
// allow it; 4-byte elements otherwise) from each of the W inputs (W independent loads in flight per lane, nontemporal since each is
// read once) and writes one vector.  int32 sums wrap modulo 2^32, like a
// switch's integer adders; fp32 adds in worker order 0..W-1 so the result
// does not depend on scheduling.
#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kBlock = 256;

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

struct AddU32 {
    typedef uint32_t S;
    typedef v4u V;
    __device__ static V op(V a, V b) { return a + b; }
    __device__ static S op(S a, S b) { return a + b; }
};
struct AddF32 {
    typedef float S;
    typedef v4f V;
    __device__ static V op(V a, V b) { return a + b; }
    __device__ static S op(S a, S b) { return a + b; }
};
struct OrU32 {
    typedef uint32_t S;
    typedef v4u V;
    __device__ static V op(V a, V b) { return a | b; }
    __device__ static S op(S a, S b) { return a | b; }
};

// out[i] = in[0*stride + i] op in[1*stride + i] op ... for i < count.
// VEC: count and stride are multiples of 4 (16-byte vectors).
template <typename OP, bool VEC>
__global__ __launch_bounds__(kBlock) void reduce_workers_kernel(
    const typename OP::S* __restrict__ in, typename OP::S* __restrict__ out, uint64_t count,
    uint64_t stride, uint32_t W) {
    typedef typename OP::S S;
    typedef typename OP::V V;
    const uint64_t step = (uint64_t)gridDim.x * kBlock;
    const uint64_t first = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    if (VEC) {
        const uint64_t nvec = count / 4, vstride = stride / 4;
        const V* vin = reinterpret_cast<const V*>(in);
        for (uint64_t i = first; i < nvec; i += step) {
            V acc = __builtin_nontemporal_load(vin + i);
            for (uint32_t w = 1; w < W; w++)
                acc = OP::op(acc, __builtin_nontemporal_load(vin + (uint64_t)w * vstride + i));
            reinterpret_cast<V*>(out)[i] = acc;
        }
    } else {
        for (uint64_t i = first; i < count; i += step) {
            S acc = __builtin_nontemporal_load(in + i);
            for (uint32_t w = 1; w < W; w++)
                acc = OP::op(acc, __builtin_nontemporal_load(in + (uint64_t)w * stride + i));
            out[i] = acc;
        }
    }
}

template <typename OP>
hipError_t launch_reduce(const void* in, void* out, uint64_t count, uint32_t W, int cus,
                         hipStream_t s) {
    typedef typename OP::S S;
    const bool vec = (count % 4) == 0 && (reinterpret_cast<uintptr_t>(in) & 15u) == 0 &&
                     (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
    const uint64_t items = vec ? count / 4 : count;
    uint64_t grid = (items + kBlock - 1) / kBlock;
    const uint64_t cap = (uint64_t)cus * 16;
    if (grid > cap) grid = cap;
    if (grid < 1) grid = 1;
    if (vec)
        hipLaunchKernelGGL((reduce_workers_kernel<OP, true>), dim3((uint32_t)grid), dim3(kBlock),
                           0, s, static_cast<const S*>(in), static_cast<S*>(out), count, count, W);
    else
        hipLaunchKernelGGL((reduce_workers_kernel<OP, false>), dim3((uint32_t)grid),
                           dim3(kBlock), 0, s, static_cast<const S*>(in), static_cast<S*>(out),
                           count, count, W);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_aggregate(const Geo& g, const void* y_in, const uint32_t* b_in, uint32_t W,
                            void* y_out, uint32_t* b_out, hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    e = g.f32 ? launch_reduce<AddF32>(y_in, y_out, g.cells, W, di.cus, s)
              : launch_reduce<AddU32>(y_in, y_out, g.cells, W, di.cus, s);
    if (e != hipSuccess) return e;
    return launch_reduce<OrU32>(b_in, b_out, g.bwords, W, di.cus, s);
}

}  // namespace hc
