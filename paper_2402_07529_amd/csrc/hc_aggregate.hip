// hc_aggregate.hip -- the aggregation step between the two phases of
// Algorithm 1, run on one GPU in place of the switch / AllReduce:
// Y <- sum over workers of Y_w, B <- OR over workers of B_w (section 3).
//
// A pure HBM stream: every lane reads 16 bytes (one vector of 4 elements,
// two of 2 or four single ones, as the buffers' alignment allows) from each
// of the W inputs (all loads in flight together, nontemporal since each is
// read once) and writes them out.  int32 sums wrap modulo 2^32, like a
// switch's integer adders; fp32 adds in worker order 0..W-1 so the result
// does not depend on scheduling.
#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kBlock = 256;

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

// op applies elementwise to scalars and to vectors of any width
struct AddU32 {
    typedef uint32_t S;
    typedef v4u V;
    template <typename X> __device__ static X op(X a, X b) { return a + b; }
};
struct AddF32 {
    typedef float S;
    typedef v4f V;
    template <typename X> __device__ static X op(X a, X b) { return a + b; }
};
struct OrU32 {
    typedef uint32_t S;
    typedef v4u V;
    template <typename X> __device__ static X op(X a, X b) { return a | b; }
};

template <typename OP, int VW> struct VecOf;
template <typename OP> struct VecOf<OP, 4> { typedef typename OP::V type; };
template <typename OP> struct VecOf<OP, 2> {
    typedef typename OP::S type __attribute__((ext_vector_type(2)));
};
template <typename OP> struct VecOf<OP, 1> { typedef typename OP::S type; };

// out[i] = in[0*stride + i] op in[1*stride + i] op ... for i < count, in
// vectors of VW elements (count, stride and both bases multiples of VW
// elements, so every worker's vectors are aligned).  Each lane takes 16 bytes
// per worker per pass: one vector of 4, two of 2, or four single elements,
// spaced a grid apart so that each wave-wide load stays contiguous; all W of
// a lane's loads are in flight together.  VGG19-sized bitmaps have an even
// word count that is not a multiple of four, so they take the pairs.
template <typename OP, int VW>
__global__ __launch_bounds__(kBlock) void reduce_workers_kernel(
    const typename OP::S* __restrict__ in, typename OP::S* __restrict__ out, uint64_t count,
    uint64_t stride, uint32_t W) {
    typedef typename VecOf<OP, VW>::type V;
    constexpr uint32_t U = 4 / VW;
    const uint64_t step = (uint64_t)gridDim.x * kBlock;
    const uint64_t first = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    const uint64_t nvec = count / VW, vstride = stride / VW;
    const V* vin = reinterpret_cast<const V*>(in);
    V* vout = reinterpret_cast<V*>(out);
    for (uint64_t i = first; i < nvec; i += step * U) {
        V acc[U];
#pragma unroll
        for (uint32_t u = 0; u < U; u++)
            if (i + u * step < nvec) acc[u] = __builtin_nontemporal_load(vin + i + u * step);
        for (uint32_t w = 1; w < W; w++) {
            const V* src = vin + (uint64_t)w * vstride + i;
#pragma unroll
            for (uint32_t u = 0; u < U; u++)
                if (i + u * step < nvec)
                    acc[u] = OP::op(acc[u], __builtin_nontemporal_load(src + u * step));
        }
#pragma unroll
        for (uint32_t u = 0; u < U; u++)
            if (i + u * step < nvec) vout[i + u * step] = acc[u];
    }
}

template <typename OP>
hipError_t launch_reduce(const void* in, void* out, uint64_t count, uint32_t W, int cus,
                         hipStream_t s) {
    typedef typename OP::S S;
    const uintptr_t al = reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out);
    const int vw = (count % 4 == 0 && (al & 15u) == 0) ? 4
                   : ((count % 2 == 0 && (al & 7u) == 0) ? 2 : 1);
    const uint64_t items = (count / vw + (4 / vw) - 1) / (4 / vw);  // lanes' passes of 16 bytes
    uint64_t grid = (items + kBlock - 1) / kBlock;
    const uint64_t cap = (uint64_t)cus * 16;
    if (grid > cap) grid = cap;
    if (grid < 1) grid = 1;
    const S* src = static_cast<const S*>(in);
    S* dst = static_cast<S*>(out);
    if (vw == 4)
        hipLaunchKernelGGL((reduce_workers_kernel<OP, 4>), dim3((uint32_t)grid), dim3(kBlock), 0, s,
                           src, dst, count, count, W);
    else if (vw == 2)
        hipLaunchKernelGGL((reduce_workers_kernel<OP, 2>), dim3((uint32_t)grid), dim3(kBlock), 0, s,
                           src, dst, count, count, W);
    else
        hipLaunchKernelGGL((reduce_workers_kernel<OP, 1>), dim3((uint32_t)grid), dim3(kBlock), 0, s,
                           src, dst, count, count, W);
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
