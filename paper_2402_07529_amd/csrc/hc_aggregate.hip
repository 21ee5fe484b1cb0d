// hc_aggregate.hip -- the aggregation step between the two phases of
// Algorithm 1, run on one GPU in place of the switch / AllReduce:
// Y <- sum over workers of Y_w, B <- OR over workers of B_w (section 3).
//
// A pure HBM stream: every lane reads 16 bytes from each of the W inputs
// (nontemporal, since each is read once) and writes the result out.  With
// 16-byte aligned buffers the 16 bytes are one aligned vector also when the
// per-worker count is not a multiple of four (the words are realigned across
// lanes); other buffers take two vectors of 2 or four single elements.  int32 sums wrap modulo 2^32, like a
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
// spaced a grid apart so that each wave-wide load stays contiguous.  The
// worker loop combines each load before the next is issued, so a lane has one
// load in flight and the occupancy keeps the stream going: issuing eight
// workers' loads before combining them measured slower on every line (BERT-base
// at 5 %, 16 workers: 1.32 -> 1.41 ms; NCF 0.207 -> 0.214 ms).  Used for 16-byte aligned buffers
// whose count is a multiple of four (VW = 4) and for buffers that are not
// 16-byte aligned (VW = 2 or 1).
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

// The same for a per-worker count that is not a multiple of four (16-byte
// aligned in and out): worker w then starts (w * count) mod 4 words past a
// 16-byte boundary.  Each lane still loads one aligned 16-byte chunk per
// worker, the one holding the first word of its output vector; the words
// past that chunk's end are the first words of the next lane's chunk, taken
// by a shuffle, or, for the wave's last lane and the last vector, loaded
// word by word.  Four workers' chunks are loaded before any is shuffled.
// Blocks loop while any lane of the wave has work (the shuffles need every
// lane); block 0 also writes the count mod 4 tail words.
template <typename OP>
__global__ __launch_bounds__(kBlock) void reduce_workers_shift_kernel(
    const typename OP::S* __restrict__ in, typename OP::S* __restrict__ out, uint64_t count,
    uint32_t W) {
    typedef typename OP::S S;
    typedef typename OP::V V;
    const uint64_t nvec = count / 4;
    const uint64_t step = (uint64_t)gridDim.x * kBlock;
    const uint32_t lane = lane_id();
    const V* vin = reinterpret_cast<const V*>(in);
    for (uint64_t i0 = (uint64_t)blockIdx.x * kBlock + (threadIdx.x & ~63u); i0 < nvec;
         i0 += step) {
        const uint64_t i = i0 + lane;
        const bool live = i < nvec;
        const bool own = live && (lane == 63u || i + 1 >= nvec);
        V acc = {};
        for (uint32_t w0 = 0; w0 < W; w0 += 4) {
            V L[4];
#pragma unroll
            for (uint32_t u = 0; u < 4; u++) {
                const uint64_t wb = (uint64_t)(w0 + u) * count;
                L[u] = (w0 + u < W && live) ? __builtin_nontemporal_load(vin + (wb >> 2) + i) : V{};
            }
#pragma unroll
            for (uint32_t u = 0; u < 4; u++) {
                if (w0 + u >= W) break;
                const uint64_t wb = (uint64_t)(w0 + u) * count;
                const uint32_t m = (uint32_t)(wb & 3u);
                S n0 = __shfl_down(L[u].x, 1), n1 = __shfl_down(L[u].y, 1),
                  n2 = __shfl_down(L[u].z, 1);
                if (own && m != 0u) {
                    const S* p = in + wb + 4 * i + 4 - m;  // words wb + 4i + 4 - m .. wb + 4i + 3
                    n0 = p[0];
                    n1 = m >= 2u ? p[1] : S(0);
                    n2 = m >= 3u ? p[2] : S(0);
                }
                const V v = m == 0u   ? L[u]
                            : m == 1u ? V{L[u].y, L[u].z, L[u].w, n0}
                            : m == 2u ? V{L[u].z, L[u].w, n0, n1}
                                      : V{L[u].w, n0, n1, n2};
                acc = (w0 + u == 0) ? v : OP::op(acc, v);
            }
        }
        if (live) reinterpret_cast<V*>(out)[i] = acc;
    }
    if (blockIdx.x == 0) {
        for (uint64_t k = 4 * nvec + threadIdx.x; k < count; k += kBlock) {
            S a = in[k];
            for (uint32_t w = 1; w < W; w++) a = OP::op(a, in[(uint64_t)w * count + k]);
            out[k] = a;
        }
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
    if (vw != 4 && (al & 15u) == 0 && count >= 4) {
        // worker strides off the 16-byte grid: aligned loads, shifted by shuffles
        const uint64_t nvec = count / 4;
        uint64_t g2 = (nvec + kBlock - 1) / kBlock;
        if (g2 > cap) g2 = cap;
        hipLaunchKernelGGL((reduce_workers_shift_kernel<OP>), dim3((uint32_t)g2), dim3(kBlock), 0,
                           s, src, dst, count, W);
    } else if (vw == 4)
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
