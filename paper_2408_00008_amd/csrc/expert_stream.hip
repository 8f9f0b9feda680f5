// Weight-streaming grouped expert GEMMs for decode shapes (few rows per
// expert), gfx950.
//
// In a decode step each active expert sees only a handful of token rows, so
// the layer is bound by reading the expert weights from HBM (arithmetic
// intensity = rows per expert flop/byte, far below the MFMA/HBM ridge).  The
// kernels therefore read every weight byte exactly once:
//
//   * a workgroup owns one expert e and a slab of 16*NS weight rows; each wave
//     of the slab owns 16 rows and a 1/KS share of the reduction dimension;
//   * weights go straight from HBM into registers as the A operand of a
//     16x16x32 bf16 MFMA (lane l reads 16 contiguous bytes of row l%16), one
//     chunk of KC reduction elements ahead of the MFMAs that consume them;
//   * the expert's token rows (<= 16*G per pass) are staged through LDS once
//     per chunk and shared by the NS waves of a reduction share (B operand);
//   * UP fuses w1 and w3 (two accumulators over the same token fragment) and
//     the SiLU*mul epilogue, writing h in bf16; DOWN fuses the gate-weighted
//     scatter of each row back to its (token, slot) position in f32;
//   * partial sums of the KS reduction shares are added in LDS in a fixed
//     order, so results are bitwise reproducible.
//
// Per-expert row counts come from the device-side offsets; experts with no
// rows exit at once and no host synchronisation is needed.  An expert with
// more than 16*G rows is processed in passes (weights re-read per pass).
#include "common.hpp"
#include "launch.hpp"

namespace moe {

namespace {

struct StreamParams {
    const bf16_t* act;       // token rows (UP: x, DOWN: h)
    const int32_t* gather;   // UP: source row = gather[r] / kslots (null = r)
    int kslots;
    const int32_t* offsets;  // [E+1]
    const bf16_t* wa;        // UP: w1, DOWN: w2   [E, N, K]
    const bf16_t* wb;        // UP: w3             [E, N, K]
    int N, K;                // weight rows / reduction length per expert
    bf16_t* h_out;           // UP   [A, N]
    float* y_out;            // DOWN [A, N]
    const float* topk_w;     // DOWN, null = unweighted row order
    const int32_t* perm;     // DOWN
};

template <bool UP, int NS, int KS, int G, int KC>
struct StreamCfg {
    static constexpr int THREADS = 64 * NS * KS;
    static constexpr int ROWS = 16 * NS;          // weight rows per workgroup
    static constexpr int MT = 16 * G;             // token rows per pass
    static constexpr int LDK = KC + 8;            // padded LDS row (bf16 elements)
    static constexpr int KSTEPS = KC / 32;        // MFMA k-steps per chunk
    static constexpr int GROUP_THREADS = 64 * NS; // threads sharing one token tile
    static constexpr int TILE_LOADS = MT * KC / 8;
    static constexpr int TPT = (TILE_LOADS + GROUP_THREADS - 1) / GROUP_THREADS;
    static constexpr int NMAT = UP ? 2 : 1;
    static constexpr int TILE_BYTES = KS * MT * LDK * 2;
    static constexpr int RED_BYTES = (KS - 1) * NS * 64 * G * 4 * NMAT * 4;
    static constexpr int LDS_BYTES = TILE_BYTES > RED_BYTES ? TILE_BYTES : RED_BYTES;
};

template <bool UP, int NS, int KS, int G, int KC>
__global__ __launch_bounds__(64 * NS * KS) void stream_kernel(StreamParams p)
{
    using C = StreamCfg<UP, NS, KS, G, KC>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::LDS_BYTES];

    const int nbn = p.N / C::ROWS;
    const int e = blockIdx.x / nbn;
    const int nb = blockIdx.x - e * nbn;
    const int row0 = p.offsets[e];
    const int M = p.offsets[e + 1] - row0;
    if (M <= 0) return;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ns = wave % NS, ks = wave / NS;
    const int gt = tid % C::GROUP_THREADS;  // index within the token-tile group
    const int n0 = nb * C::ROWS + ns * 16;
    const int kper = p.K / KS;
    const int kbeg = ks * kper;
    const int nchunks = kper / KC;

    bf16_t* tile = reinterpret_cast<bf16_t*>(smem) + ks * C::MT * C::LDK;

    const int64_t wrow = (int64_t)e * p.N + n0 + (lane & 15);
    const bf16_t* pa = p.wa + wrow * p.K + kbeg + 8 * (lane >> 4);
    const bf16_t* pb = UP ? p.wb + wrow * p.K + kbeg + 8 * (lane >> 4) : nullptr;

    for (int m0 = 0; m0 < M; m0 += C::MT) {
        const int Mp = min(M - m0, C::MT);
        const int gact = (Mp + 15) >> 4;

        // source row pointer of each 16-byte staging load of this thread
        const bf16_t* src[C::TPT];
        int ldsoff[C::TPT];
        bool live[C::TPT];
#pragma unroll
        for (int it = 0; it < C::TPT; ++it) {
            const int q = it * C::GROUP_THREADS + gt;
            live[it] = q < C::TILE_LOADS;
            const int m = live[it] ? q / (KC / 8) : 0;
            const int c8 = live[it] ? q % (KC / 8) : 0;
            const int mm = m < Mp ? m : Mp - 1;  // rows past the end repeat the last row
            const int r = row0 + m0 + mm;
            const int64_t sr = (UP && p.gather) ? p.gather[r] / p.kslots : r;
            src[it] = p.act + sr * p.K + kbeg + c8 * 8;
            ldsoff[it] = m * C::LDK + c8 * 8;
        }

        floatx4 accA[G], accB[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            accA[g] = floatx4{0.f, 0.f, 0.f, 0.f};
            accB[g] = floatx4{0.f, 0.f, 0.f, 0.f};
        }

        uint4 treg[C::TPT];
        bf16x8 wA[C::KSTEPS], wB[C::KSTEPS];
#pragma unroll
        for (int it = 0; it < C::TPT; ++it)
            if (live[it]) treg[it] = ldg16(src[it]);
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk) {
            wA[kk] = as_bf16x8(ldg16(pa + kk * 32));
            if (UP) wB[kk] = as_bf16x8(ldg16(pb + kk * 32));
        }

        for (int c = 0; c < nchunks; ++c) {
            __syncthreads();
#pragma unroll
            for (int it = 0; it < C::TPT; ++it)
                if (live[it]) *reinterpret_cast<uint4*>(tile + ldsoff[it]) = treg[it];
            bf16x8 nA[C::KSTEPS], nB[C::KSTEPS];
            if (c + 1 < nchunks) {
                const int ko = (c + 1) * KC;
#pragma unroll
                for (int it = 0; it < C::TPT; ++it)
                    if (live[it]) treg[it] = ldg16(src[it] + ko);
#pragma unroll
                for (int kk = 0; kk < C::KSTEPS; ++kk) {
                    nA[kk] = as_bf16x8(ldg16(pa + ko + kk * 32));
                    if (UP) nB[kk] = as_bf16x8(ldg16(pb + ko + kk * 32));
                }
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < C::KSTEPS; ++kk) {
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    if (g < gact) {
                        const bf16x8 b = *reinterpret_cast<const bf16x8*>(
                            tile + (g * 16 + (lane & 15)) * C::LDK + kk * 32 + 8 * (lane >> 4));
                        accA[g] = mfma16x16x32(wA[kk], b, accA[g]);
                        if (UP) accB[g] = mfma16x16x32(wB[kk], b, accB[g]);
                    }
                }
            }
            if (c + 1 < nchunks) {
#pragma unroll
                for (int kk = 0; kk < C::KSTEPS; ++kk) {
                    wA[kk] = nA[kk];
                    if (UP) wB[kk] = nB[kk];
                }
            }
        }

        if (KS > 1) {
            // add the reduction shares ks = 1..KS-1 into share 0, in order
            __syncthreads();
            float* red = reinterpret_cast<float*>(smem);
            if (ks > 0) {
                float* dst = red + ((ks - 1) * NS + ns) * (64 * G * 4 * C::NMAT);
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    if (g < gact) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            dst[((g * 4 + i) * C::NMAT + 0) * 64 + lane] = accA[g][i];
                            if (UP) dst[((g * 4 + i) * C::NMAT + 1) * 64 + lane] = accB[g][i];
                        }
                    }
                }
            }
            __syncthreads();
            if (ks == 0) {
                for (int s = 1; s < KS; ++s) {
                    const float* srcr = red + ((s - 1) * NS + ns) * (64 * G * 4 * C::NMAT);
#pragma unroll
                    for (int g = 0; g < G; ++g) {
                        if (g < gact) {
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                accA[g][i] += srcr[((g * 4 + i) * C::NMAT + 0) * 64 + lane];
                                if (UP) accB[g][i] += srcr[((g * 4 + i) * C::NMAT + 1) * 64 + lane];
                            }
                        }
                    }
                }
            }
        }

        if (ks == 0) {
            const int n = n0 + 4 * (lane >> 4);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const int tok = g * 16 + (lane & 15);
                if (g < gact && tok < Mp) {
                    const int64_t r = row0 + m0 + tok;
                    if (UP) {
                        uint2 pk;
                        pk.x = pack_bf16x2(silu(accA[g][0]) * accB[g][0],
                                           silu(accA[g][1]) * accB[g][1]);
                        pk.y = pack_bf16x2(silu(accA[g][2]) * accB[g][2],
                                           silu(accA[g][3]) * accB[g][3]);
                        *reinterpret_cast<uint2*>(p.h_out + r * p.N + n) = pk;
                    } else {
                        int64_t orow = r;
                        float gw = 1.0f;
                        if (p.topk_w && p.perm) {
                            orow = p.perm[r];
                            gw = p.topk_w[orow];
                        }
                        float4 v;
                        v.x = gw * accA[g][0];
                        v.y = gw * accA[g][1];
                        v.z = gw * accA[g][2];
                        v.w = gw * accA[g][3];
                        *reinterpret_cast<float4*>(p.y_out + orow * p.N + n) = v;
                    }
                }
            }
        }
    }
}

template <bool UP, int NS, int KS, int G, int KC>
hipError_t run(const StreamParams& p, int E, hipStream_t stream)
{
    using C = StreamCfg<UP, NS, KS, G, KC>;
    const unsigned grid = static_cast<unsigned>(E * (p.N / C::ROWS));
    stream_kernel<UP, NS, KS, G, KC><<<grid, C::THREADS, 0, stream>>>(p);
    return hipGetLastError();
}

int groups_for(int64_t rows_max)
{
    if (rows_max <= 16) return 1;
    if (rows_max <= 32) return 2;
    if (rows_max <= 64) return 4;
    if (rows_max <= 128) return 8;
    return 16;
}

template <bool UP, int NS, int KS, int KC>
hipError_t run_g(const StreamParams& p, int E, int G, hipStream_t stream)
{
    switch (G) {
    case 1: return run<UP, NS, KS, 1, KC>(p, E, stream);
    case 2: return run<UP, NS, KS, 2, KC>(p, E, stream);
    case 4: return run<UP, NS, KS, 4, KC>(p, E, stream);
    default: return hipErrorInvalidValue;
    }
}

template <bool UP, int NS, int KS>
hipError_t run_g_big(const StreamParams& p, int E, int G, hipStream_t stream)
{
    // large token tiles use 64-element chunks to bound registers and LDS
    switch (G) {
    case 8: return run<UP, NS, KS, 8, 64>(p, E, stream);
    case 16: return run<UP, NS, KS, 16, 64>(p, E, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

// Rows of one expert are at most T (each token picks distinct experts), and
// at most A = T*k.  Tokens per expert pass: 16*G.
hipError_t launch_stream_up(const UpArgs& a, int64_t rows_max, hipStream_t stream)
{
    StreamParams p{};
    p.act = a.x;
    p.gather = a.gather;
    p.kslots = a.kslots;
    p.offsets = a.offsets;
    p.wa = a.w1;
    p.wb = a.w3;
    p.N = a.ffn;
    p.K = a.d;
    p.h_out = a.h;
    const int G = groups_for(rows_max);
    if (G >= 8) return run_g_big<true, 4, 1>(p, a.E, G, stream);
    if (a.d % 128 == 0) return run_g<true, 4, 1, 128>(p, a.E, G, stream);
    return run_g<true, 4, 1, 64>(p, a.E, G, stream);
}

hipError_t launch_stream_down(const DownArgs& a, int64_t rows_max, hipStream_t stream)
{
    StreamParams p{};
    p.act = a.h;
    p.offsets = a.offsets;
    p.wa = a.w2;
    p.N = a.d;
    p.K = a.ffn;
    p.y_out = a.y;
    p.topk_w = a.topk_w;
    p.perm = a.perm;
    const int G = groups_for(rows_max);
    if (G >= 8) {
        if (a.ffn % 128 == 0) return run_g_big<false, 2, 2>(p, a.E, G, stream);
        return run_g_big<false, 4, 1>(p, a.E, G, stream);
    }
    if (a.ffn % 256 == 0) return run_g<false, 2, 2, 128>(p, a.E, G, stream);
    if (a.ffn % 128 == 0) return run_g<false, 2, 2, 64>(p, a.E, G, stream);
    return run_g<false, 4, 1, 64>(p, a.E, G, stream);
}

}  // namespace moe
