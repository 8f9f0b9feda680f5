// Row gather, slot combine and RMSNorm for gfx950: HBM-bound copies, written
// as grid-stride loops of 16-byte vector accesses so consecutive lanes touch
// consecutive bytes of a row.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

namespace {

// x_perm[r,:] = x[perm[r] / k, :]
__global__ __launch_bounds__(256) void permute_kernel(const bf16_t* __restrict__ x,
                                                      const int32_t* __restrict__ perm, int64_t A,
                                                      int d, int k, bf16_t* __restrict__ x_perm)
{
    const int cpr = d >> 3;  // 16-byte chunks per row
    const int64_t total = A * cpr;
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = q / cpr;
        const int c = static_cast<int>(q - r * cpr);
        const int64_t t = perm[r] / k;
        *reinterpret_cast<uint4*>(x_perm + r * d + c * 8) = ldg16(x + t * d + c * 8);
    }
}

// s = residual + sum_{j ascending} y[t*k+j]; out = bf16(s), out_f32 = s
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ y,
                                                      const float* residual, int64_t T, int d,
                                                      int k, const int* nslices,
                                                      int max_slices, bf16_t* __restrict__ out,
                                                      float* out_f32)
{
    const int cpr = d >> 2;  // float4 per row
    const int64_t total = T * cpr;
    // y may hold the partial sums of several reduction parts, slice s at
    // y + s * T * k * d; each slot sums its slices in ascending order
    const int ns = nslices ? min(max(*nslices, 1), max_slices) : 1;
    const int64_t slice = T * k * d;
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t t = q / cpr;
        const int c = static_cast<int>(q - t * cpr);
        float4 s = residual ? *reinterpret_cast<const float4*>(residual + t * d + c * 4)
                            : make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j = 0; j < k; ++j) {
            const float* yj = y + (t * k + j) * d + c * 4;
            float4 v = *reinterpret_cast<const float4*>(yj);
            for (int q = 1; q < ns; ++q) {
                const float4 u = *reinterpret_cast<const float4*>(yj + q * slice);
                v.x += u.x;
                v.y += u.y;
                v.z += u.z;
                v.w += u.w;
            }
            s.x += v.x;
            s.y += v.y;
            s.z += v.z;
            s.w += v.w;
        }
        if (out) {
            uint2 p;
            p.x = pack_bf16x2(s.x, s.y);
            p.y = pack_bf16x2(s.z, s.w);
            *reinterpret_cast<uint2*>(out + t * d + c * 4) = p;
        }
        if (out_f32) *reinterpret_cast<float4*>(out_f32 + t * d + c * 4) = s;
    }
}

// a = bf16(h * rsqrt(mean(h^2) + eps) * gamma), one workgroup per row
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ h,
                                                      const bf16_t* __restrict__ gamma, int64_t T,
                                                      int d, float eps, bf16_t* __restrict__ a)
{
    __shared__ float red[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
        const float* hr = h + t * d;
        float ss = 0.0f;
        for (int c = tid; c < (d >> 2); c += 256) {
            const float4 v = *reinterpret_cast<const float4*>(hr + c * 4);
            ss = fmaf(v.x, v.x, ss);
            ss = fmaf(v.y, v.y, ss);
            ss = fmaf(v.z, v.z, ss);
            ss = fmaf(v.w, v.w, ss);
        }
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
        if (lane == 0) red[wave] = ss;
        __syncthreads();
        const float tot = (red[0] + red[1]) + (red[2] + red[3]);
        const float inv = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
        for (int c = tid; c < (d >> 2); c += 256) {
            const float4 v = *reinterpret_cast<const float4*>(hr + c * 4);
            const uint2 g = *reinterpret_cast<const uint2*>(gamma + c * 4);
            uint2 p;
            p.x = pack_bf16x2(v.x * inv * __uint_as_float(g.x << 16),
                              v.y * inv * __uint_as_float(g.x & 0xffff0000u));
            p.y = pack_bf16x2(v.z * inv * __uint_as_float(g.y << 16),
                              v.w * inv * __uint_as_float(g.y & 0xffff0000u));
            *reinterpret_cast<uint2*>(a + t * d + c * 4) = p;
        }
        __syncthreads();
    }
}

unsigned grid_for(int64_t work, int threads)
{
    int64_t b = (work + threads - 1) / threads;
    if (b > 65536) b = 65536;
    return static_cast<unsigned>(b < 1 ? 1 : b);
}

}  // namespace

hipError_t launch_permute(const bf16_t* x, const int32_t* perm, int64_t A, int d, int k,
                          bf16_t* x_perm, hipStream_t stream)
{
    if (A == 0) return hipSuccess;
    permute_kernel<<<grid_for(A * (d / 8), 256), 256, 0, stream>>>(x, perm, A, d, k, x_perm);
    return hipGetLastError();
}

hipError_t launch_combine(const float* y, const float* residual, int64_t T, int d, int k,
                          bf16_t* out, float* out_f32, hipStream_t stream, const int* nslices,
                          int max_slices)
{
    if (T == 0) return hipSuccess;
    combine_kernel<<<grid_for(T * (d / 4), 256), 256, 0, stream>>>(y, residual, T, d, k, nslices,
                                                                   max_slices, out, out_f32);
    return hipGetLastError();
}

// After the tiled down GEMM over the experts with at least mlo rows ran with
// its reduction cut: slice 0 of each of their rows += slices 1 .. n-1 in
// ascending order (the order the combine uses).  n is recomputed here with the
// cost model that kernel used (same tile count, grid, steps, sizes and cap),
// so the count needs no device handoff; *parts_out (if not null) is set to 1
// for the combine.  Permuted row r lives at y row perm[r] (perm null: r).
// Blocks take (row, 1024-column chunk) units.
__global__ __launch_bounds__(256) void fold_parts_kernel(float* __restrict__ y, int64_t A, int d,
                                                         const int32_t* __restrict__ offsets,
                                                         int E, int mlo,
                                                         const int32_t* __restrict__ perm,
                                                         int nk, int per_xcd, int smax,
                                                         int* parts_out)
{
    if (parts_out && blockIdx.x == 0 && threadIdx.x == 0) *parts_out = 1;
    int tiles = 0;
    for (int e = 0; e < E; ++e) {
        const int m = offsets[e + 1] - offsets[e];
        if (m >= mlo) tiles += (m + 255) >> 8;
    }
    const int ns = down_parts((d >> 8) * tiles, per_xcd, nk, A, d, smax);
    if (ns <= 1) return;
    const int64_t slice = A * d;
    const int cpr = d >> 2;                  // float4 per row
    const int chunks = (cpr + 255) >> 8;     // 256 float4 per unit
    for (int64_t u = blockIdx.x; u < A * chunks; u += gridDim.x) {
        const int64_t r = u / chunks;
        const int c = static_cast<int>(u - r * chunks) * 256 + threadIdx.x;
        // the expert holding row r: offsets are non-decreasing with offsets[E] = A
        int e = 0;
        while (e + 1 < E && offsets[e + 1] <= r) ++e;
        if (offsets[e + 1] - offsets[e] < mlo || c >= cpr) continue;
        float4* y0 = reinterpret_cast<float4*>(y + (perm ? (int64_t)perm[r] : r) * d) + c;
        float4 v = *y0;
        // loads four slices at a time, adds them in order
        for (int q = 1; q < ns; q += 4) {
            float4 t[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (q + i < ns) t[i] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(y0) + (q + i) * slice);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (q + i < ns) {
                    v.x += t[i].x;
                    v.y += t[i].y;
                    v.z += t[i].z;
                    v.w += t[i].w;
                }
        }
        *y0 = v;
    }
}

hipError_t launch_fold_parts(float* y, int64_t A, int d, const int32_t* offsets, int E, int mlo,
                             const int32_t* perm, int nk, int per_xcd, int smax, int* parts_out,
                             hipStream_t stream)
{
    if (A == 0) return hipSuccess;
    const int64_t units = A * (((d >> 2) + 255) >> 8);
    const unsigned grid = static_cast<unsigned>(units < 8192 ? units : 8192);
    fold_parts_kernel<<<grid, 256, 0, stream>>>(y, A, d, offsets, E, mlo, perm, nk, per_xcd, smax,
                                                parts_out);
    return hipGetLastError();
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v) { *p = v; }

hipError_t launch_fill_i32(int32_t* p, int32_t v, hipStream_t stream)
{
    fill_i32_kernel<<<1, 1, 0, stream>>>(p, v);
    return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* h, const bf16_t* gamma, int64_t T, int d, float eps,
                          bf16_t* a, hipStream_t stream)
{
    if (T == 0) return hipSuccess;
    const unsigned grid = static_cast<unsigned>(T < 65536 ? T : 65536);
    rmsnorm_kernel<<<grid, 256, 0, stream>>>(h, gamma, T, d, eps, a);
    return hipGetLastError();
}

}  // namespace moe
