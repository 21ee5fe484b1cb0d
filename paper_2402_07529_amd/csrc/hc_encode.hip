// hc_encode.hip -- worker-side compression (Algorithm 1, phase I) for gfx950.
//
// Dense path.  A workgroup of 256 lanes takes tiles of 1024 consecutive
// parameters; each lane loads four with one 16-byte nontemporal load (the
// gradient is read once, so it should not evict the sketch from L2/MALL).
// Per wave (256 parameters):
//   - four ballots of "x != 0" become the eight bitmap words of the wave
//     (section 3.2), written by lanes 0..7;
//   - every nonzero adds g_j * x to its three cells (section 3.1) with
//     fire-and-forget global atomics.  Within one batch the cells of a hash
//     are one sketch row rotated by a bias (section 3.4), so the atomics of a
//     wave land in at most three 4 KiB rows.
// The batch hash is wave-uniform when c >= 256 (computed on the scalar unit
// once per wave and tile), per lane when 4 <= c < 256, per element below.
#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kBlock = 256;
constexpr uint64_t kTile = 1024;  // parameters per workgroup and iteration

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

template <typename T> struct Vec4;
template <> struct Vec4<int32_t> { typedef v4i type; };
template <> struct Vec4<float> { typedef v4f type; };

// vec: p is 16-byte aligned (else plain 4-byte stores throughout).
__global__ __launch_bounds__(kBlock) void fill_u32_kernel(uint32_t* __restrict__ p,
                                                          uint64_t count, uint32_t value,
                                                          bool vec) {
    const uint64_t nvec = vec ? count / 4 : 0;
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    if (!vec) {
        for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
            p[i] = value;
        return;
    }
    const v4u v = {value, value, value, value};
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < nvec; i += stride)
        reinterpret_cast<v4u*>(p)[i] = v;
    if (blockIdx.x == 0 && threadIdx.x < count - nvec * 4) p[nvec * 4 + threadIdx.x] = value;
}

// MODE 0: c >= 256, MODE 1: 4 <= c < 256, MODE 2: c < 4.
template <typename T, int MODE>
__global__ __launch_bounds__(kBlock) void encode_dense_kernel(
    const T* __restrict__ x, T* __restrict__ y, uint32_t* __restrict__ b, uint64_t n,
    uint64_t words, uint64_t seed, uint32_t rows, uint32_t c, uint32_t cmask, uint32_t log2c,
    bool vec) {
    typedef typename Vec4<T>::type V;
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    const uint64_t ntiles = (n + kTile - 1) / kTile;

    for (uint64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const uint64_t base = tile * kTile + (uint64_t)wave * 256;  // wave's first parameter
        const uint64_t p0 = base + 4ull * lane;                      // lane's first parameter
        T e[4];
        if (vec && tile * kTile + kTile <= n) {
            const V v = __builtin_nontemporal_load(reinterpret_cast<const V*>(x + p0));
            e[0] = v.x; e[1] = v.y; e[2] = v.z; e[3] = v.w;
        } else {
#pragma unroll
            for (int k = 0; k < 4; k++) e[k] = (p0 + k < n) ? x[p0 + k] : T(0);
        }
        bool nz[4];
#pragma unroll
        for (int k = 0; k < 4; k++) nz[k] = Val<T>::nonzero(e[k]);

        // bitmap: element 4l+k of the wave is bit l of ballot k
        const uint64_t m0 = __ballot(nz[0]), m1 = __ballot(nz[1]);
        const uint64_t m2 = __ballot(nz[2]), m3 = __ballot(nz[3]);
        if (base < n && lane < 8) {
            const uint32_t sh = 8u * lane;
            const uint32_t word = spread4((uint32_t)(m0 >> sh)) |
                                  (spread4((uint32_t)(m1 >> sh)) << 1) |
                                  (spread4((uint32_t)(m2 >> sh)) << 2) |
                                  (spread4((uint32_t)(m3 >> sh)) << 3);
            const uint64_t widx = (base >> 5) + lane;
            if (widx < words) b[widx] = word;
        }
        if ((m0 | m1 | m2 | m3) == 0) continue;

        if (MODE == 0) {
            const BatchHash h = batch_hash(seed, rows, cmask, uniform64(base >> log2c));
            if (nz[0] | nz[1] | nz[2] | nz[3]) {
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    if (!nz[k]) continue;
                    const uint32_t t = (uint32_t)(p0 + k) & cmask;
#pragma unroll
                    for (int j = 0; j < 3; j++)
                        Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask),
                                           Val<T>::sign(e[k], (h.neg >> j) & 1u));
                }
            }
        } else if (MODE == 1) {
            if (nz[0] | nz[1] | nz[2] | nz[3]) {
                const BatchHash h = batch_hash(seed, rows, cmask, p0 >> log2c);
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    if (!nz[k]) continue;
                    const uint32_t t = (uint32_t)(p0 + k) & cmask;
#pragma unroll
                    for (int j = 0; j < 3; j++)
                        Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask),
                                           Val<T>::sign(e[k], (h.neg >> j) & 1u));
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < 4; k++) {
                if (!nz[k]) continue;
                const uint64_t p = p0 + k;
                const BatchHash h = batch_hash(seed, rows, cmask, p >> log2c);
                const uint32_t t = (uint32_t)p & cmask;
#pragma unroll
                for (int j = 0; j < 3; j++)
                    Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask),
                                       Val<T>::sign(e[k], (h.neg >> j) & 1u));
            }
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kBlock) void encode_coo_kernel(
    const uint32_t* __restrict__ idx, const T* __restrict__ val, uint64_t nnz,
    T* __restrict__ y, uint32_t* __restrict__ b, uint64_t n, uint64_t seed, uint32_t rows,
    uint32_t c, uint32_t cmask, uint32_t log2c) {
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < nnz; i += stride) {
        const uint32_t p = idx[i];
        const T v = val[i];
        if (p >= n || !Val<T>::nonzero(v)) continue;
        atomicOr(b + (p >> 5), 1u << (p & 31u));
        const BatchHash h = batch_hash(seed, rows, cmask, (uint64_t)(p >> log2c));
        const uint32_t t = p & cmask;
#pragma unroll
        for (int j = 0; j < 3; j++)
            Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask), Val<T>::sign(v, (h.neg >> j) & 1u));
    }
}

uint32_t grid_for(uint64_t work_items, uint64_t per_block, uint32_t cap) {
    uint64_t g = (work_items + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (uint32_t)g;
}

template <typename T, int MODE>
hipError_t launch_dense_t(const Geo& g, const void* x, void* y, uint32_t* b, hipStream_t s,
                          uint32_t grid) {
    hipLaunchKernelGGL((encode_dense_kernel<T, MODE>), dim3(grid), dim3(kBlock), 0, s,
                       static_cast<const T*>(x), static_cast<T*>(y), b, g.n, g.words, g.seed,
                       g.rows, g.c, g.cmask, g.log2c,
                       (reinterpret_cast<uintptr_t>(x) & 15u) == 0);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fill_u32(uint32_t* p, uint64_t count, uint32_t value, hipStream_t s) {
    if (count == 0) return hipSuccess;
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    const uint32_t grid = grid_for(count / 4 + 1, kBlock, (uint32_t)di.cus * 16);
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid), dim3(kBlock), 0, s, p, count, value,
                       (reinterpret_cast<uintptr_t>(p) & 15u) == 0);
    return hipGetLastError();
}

hipError_t launch_encode_dense(const Geo& g, const void* x, void* y, uint32_t* b,
                               hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    e = launch_fill_u32(static_cast<uint32_t*>(y), g.cells, 0u, s);
    if (e != hipSuccess) return e;
    const uint32_t grid = grid_for((g.n + kTile - 1) / kTile, 1, (uint32_t)di.cus * 8);
    const int mode = g.c >= 256 ? 0 : (g.c >= 4 ? 1 : 2);
    if (g.f32) {
        if (mode == 0) return launch_dense_t<float, 0>(g, x, y, b, s, grid);
        if (mode == 1) return launch_dense_t<float, 1>(g, x, y, b, s, grid);
        return launch_dense_t<float, 2>(g, x, y, b, s, grid);
    }
    if (mode == 0) return launch_dense_t<int32_t, 0>(g, x, y, b, s, grid);
    if (mode == 1) return launch_dense_t<int32_t, 1>(g, x, y, b, s, grid);
    return launch_dense_t<int32_t, 2>(g, x, y, b, s, grid);
}

hipError_t launch_encode_coo(const Geo& g, const uint32_t* idx, const void* val, uint64_t nnz,
                             void* y, uint32_t* b, hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    e = launch_fill_u32(static_cast<uint32_t*>(y), g.cells, 0u, s);
    if (e != hipSuccess) return e;
    e = launch_fill_u32(b, g.words, 0u, s);
    if (e != hipSuccess) return e;
    if (nnz == 0) return hipSuccess;
    const uint32_t grid = grid_for(nnz, kBlock, (uint32_t)di.cus * 16);
    if (g.f32)
        hipLaunchKernelGGL(encode_coo_kernel<float>, dim3(grid), dim3(kBlock), 0, s, idx,
                           static_cast<const float*>(val), nnz, static_cast<float*>(y), b, g.n,
                           g.seed, g.rows, g.c, g.cmask, g.log2c);
    else
        hipLaunchKernelGGL(encode_coo_kernel<int32_t>, dim3(grid), dim3(kBlock), 0, s, idx,
                           static_cast<const int32_t*>(val), nnz, static_cast<int32_t*>(y), b,
                           g.n, g.seed, g.rows, g.c, g.cmask, g.log2c);
    return hipGetLastError();
}

}  // namespace hc
