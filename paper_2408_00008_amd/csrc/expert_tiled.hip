// Tiled grouped expert GEMMs for prefill shapes (many rows per expert), gfx950.
//
// With ~1000 token rows per expert the expert FFN is MFMA-bound (arithmetic
// intensity ~ rows per expert flop/byte, above the MI355X ridge of ~310), so
// the kernels reuse both operands from LDS:
//
//   * a workgroup computes a BN x BM tile of the output (BN weight rows x BM
//     token rows) with 32x32x16 bf16 MFMAs, f32 accumulation; its 8 waves are
//     arranged WAVES_N x WAVES_M, each owning NT x MT tiles of 32x32;
//   * both operand tiles of a 64-wide reduction step are staged through LDS
//     (rows padded by 16 bytes so the 16-byte fragment reads of 16 lanes hit
//     all 64 banks once), double-buffered: the global loads of step k+1 are in
//     flight while step k is multiplied, one barrier per step;
//   * UP pairs, in each wave, 32 rows of w1 with the same 32 rows of w3, so the
//     two accumulators of an output element sit in the same lane and the
//     SiLU*mul epilogue needs no data movement; token rows are gathered
//     through the dispatch permutation while staging (no separate permute);
//   * DOWN scales each output row by its gate weight and scatters it to the
//     row's (token, slot) position;
//   * workgroups are persistent: one per CU, each walking a contiguous share
//     of the (expert, weight block, token tile) items of its XCD.  Items are
//     ordered expert, weight block, token tile, so the workgroups of one XCD
//     work on the token tiles of a few weight blocks at a time and share both
//     operands through that XCD's L2.  Per-expert tile counts are read from
//     the device-side offsets: ragged row counts need no host synchronisation.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

namespace {

struct TiledParams {
    const bf16_t* act;       // token rows (UP: x, DOWN: h)
    const int32_t* gather;   // UP: source row = gather[r] / kslots (null = r)
    int kslots;
    const int32_t* offsets;  // [E+1]
    const bf16_t* wa;        // UP: w1, DOWN: w2  [E, N, K]
    const bf16_t* wb;        // UP: w3            [E, N, K]
    int N, K, E;             // N = weight rows per expert (UP: ffn, DOWN: d)
    bf16_t* h_out;           // UP   [A, N]
    float* y_out;            // DOWN [A, N]
    const float* topk_w;     // DOWN, null = unweighted row order
    const int32_t* perm;     // DOWN
};

template <bool UP, int WAVES_N, int WAVES_M, int NT, int MT>
struct TiledCfg {
    static constexpr int THREADS = 64 * WAVES_N * WAVES_M;
    static constexpr int BN = WAVES_N * NT * 32;  // weight rows staged per workgroup
    static constexpr int BM = WAVES_M * MT * 32;  // token rows per workgroup
    static constexpr int NOUT = UP ? BN / 2 : BN; // output columns per workgroup
    static constexpr int BK = 64;
    static constexpr int LDK = BK + 8;            // padded LDS row, bf16 elements
    static constexpr int A_ELEMS = BN * LDK;
    static constexpr int STAGE_ELEMS = (BN + BM) * LDK;
    static constexpr int LDS_BYTES = 2 * STAGE_ELEMS * 2;
    static constexpr int A_LOADS = BN * BK / 8 / THREADS;
    static constexpr int B_LOADS = BM * BK / 8 / THREADS;
    static_assert(BN * BK / 8 % THREADS == 0 && BM * BK / 8 % THREADS == 0, "tile/threads");
    static_assert(!UP || (A_LOADS % 2 == 0 && (A_LOADS / 2) * (THREADS / 8) == BN / 2),
                  "UP: the first half of the A loads covers the w1 rows");
    static_assert(!UP || NT % 2 == 0, "UP pairs each w1 tile with a w3 tile per wave");
};

template <bool UP, int WAVES_N, int WAVES_M, int NT, int MT>
__global__ __launch_bounds__(64 * WAVES_N * WAVES_M) void tiled_kernel(TiledParams p)
{
    using C = TiledCfg<UP, WAVES_N, WAVES_M, NT, MT>;
    extern __shared__ __attribute__((aligned(16))) bf16_t lds[];
    __shared__ int s_items[65];  // items before expert e: nbn * (tiles of experts < e)
    __shared__ int s_tiles[65];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wn = wave % WAVES_N, wm = wave / WAVES_N;
    const int nbn = p.N / C::NOUT;

    if (tid < p.E) {
        const int M = p.offsets[tid + 1] - p.offsets[tid];
        s_tiles[tid + 1] = (M + C::BM - 1) / C::BM;
    }
    __syncthreads();
    if (tid == 0) {
        int tiles = 0;
        for (int e = 0; e < p.E; ++e) {
            s_items[e] = nbn * tiles;
            const int mt = s_tiles[e + 1];
            s_tiles[e] = tiles;
            tiles += mt;
        }
        s_items[p.E] = nbn * tiles;
        s_tiles[p.E] = tiles;
    }
    __syncthreads();
    const int total = s_items[p.E];

    // this XCD's contiguous share of the items (workgroups are handed to the
    // 8 XCDs round-robin; the grid is a multiple of 8)
    const int xcd = blockIdx.x & 7;
    const int per_xcd = gridDim.x >> 3;
    const int local = blockIdx.x >> 3;
    const int beg = (int)((int64_t)total * xcd / 8);
    const int end = (int)((int64_t)total * (xcd + 1) / 8);

    const int nk = p.K / C::BK;

    for (int w = beg + local; w < end; w += per_xcd) {
        int e = 0;
        while (s_items[e + 1] <= w) ++e;
        const int mt_e = s_tiles[e + 1] - s_tiles[e];
        const int r = w - s_items[e];
        const int nb = r / mt_e;
        const int mtile = r - nb * mt_e;
        const int row0 = p.offsets[e];
        const int M = p.offsets[e + 1] - row0;
        const int m0 = mtile * C::BM;
        const int Mp = min(C::BM, M - m0);

        // global sources of this thread's 16-byte staging loads: load `it`
        // covers tile row it * (THREADS/8) + tid/8, 16-byte column tid % 8
        constexpr int RSTEP = C::THREADS / 8;
        const int trow = tid >> 3, c8 = tid & 7;
        const bf16_t* abase1;
        const bf16_t* abase3 = nullptr;
        if (UP) {
            abase1 = p.wa + ((int64_t)e * p.N + nb * C::NOUT + trow) * p.K + c8 * 8;
            abase3 = p.wb + ((int64_t)e * p.N + nb * C::NOUT + trow) * p.K + c8 * 8;
        } else {
            abase1 = p.wa + ((int64_t)e * p.N + nb * C::NOUT + trow) * p.K + c8 * 8;
        }
        int bsrc[C::B_LOADS];  // source token row of each B load
#pragma unroll
        for (int it = 0; it < C::B_LOADS; ++it) {
            const int mm = it * RSTEP + trow;
            const int rowm = row0 + m0 + (mm < Mp ? mm : Mp - 1);
            bsrc[it] = (UP && p.gather) ? p.gather[rowm] / p.kslots : rowm;
        }
        auto a_ptr = [&](int it) -> const bf16_t* {
            if (UP) {
                constexpr int HALF = C::A_LOADS / 2;  // loads of w1 rows, then of w3 rows
                return it < HALF ? abase1 + (int64_t)it * RSTEP * p.K
                                 : abase3 + (int64_t)(it - HALF) * RSTEP * p.K;
            }
            return abase1 + (int64_t)it * RSTEP * p.K;
        };
        auto a_off = [&](int it) { return (it * RSTEP + trow) * C::LDK + c8 * 8; };
        auto b_off = [&](int it) { return C::A_ELEMS + (it * RSTEP + trow) * C::LDK + c8 * 8; };

        floatx16 acc[NT][MT];
#pragma unroll
        for (int i = 0; i < NT; ++i)
#pragma unroll
            for (int j = 0; j < MT; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

        uint4 ra[C::A_LOADS], rb[C::B_LOADS];
        auto gload = [&](int kt) {
            const int ko = kt * C::BK;
#pragma unroll
            for (int it = 0; it < C::A_LOADS; ++it) ra[it] = ldg16(a_ptr(it) + ko);
#pragma unroll
            for (int it = 0; it < C::B_LOADS; ++it)
                rb[it] = ldg16(p.act + (int64_t)bsrc[it] * p.K + c8 * 8 + ko);
        };
        auto lstore = [&](int buf) {
            bf16_t* s = lds + buf * C::STAGE_ELEMS;
#pragma unroll
            for (int it = 0; it < C::A_LOADS; ++it) *reinterpret_cast<uint4*>(s + a_off(it)) = ra[it];
#pragma unroll
            for (int it = 0; it < C::B_LOADS; ++it) *reinterpret_cast<uint4*>(s + b_off(it)) = rb[it];
        };

        // LDS row of this wave's nt-th 32-row weight tile.  UP: tiles nt < NT/2
        // are w1 rows, tile nt + NT/2 holds the same rows of w3.
        auto arow = [&](int nt) {
            if (UP) {
                constexpr int H = NT / 2;
                return (nt < H ? 0 : C::BN / 2) + wn * H * 32 + (nt % H) * 32;
            }
            return wn * NT * 32 + nt * 32;
        };

        constexpr int KSUB = C::BK / 16;  // MFMA k-steps per LDS stage
        bf16x8 fa[2][NT], fb[2][MT];      // fragments of two consecutive k-steps
        auto fread = [&](const bf16_t* s, int ks, bf16x8* a, bf16x8* b) {
            const int col = ks * 16 + 8 * (lane >> 5);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                a[nt] = *reinterpret_cast<const bf16x8*>(s + (arow(nt) + (lane & 31)) * C::LDK + col);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                b[mt] = *reinterpret_cast<const bf16x8*>(
                    s + C::A_ELEMS + (wm * MT * 32 + mt * 32 + (lane & 31)) * C::LDK + col);
        };

        gload(0);
        lstore(0);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const int buf = kt & 1;
            const bf16_t* s = lds + buf * C::STAGE_ELEMS;
            fread(s, 0, fa[0], fb[0]);
            gload(kt + 1 < nk ? kt + 1 : kt);  // unconditional: keeps the waits exact
#pragma unroll
            for (int ks = 0; ks < KSUB; ++ks) {
                const int cur = ks & 1;
                // fragments of k-step ks+1 are read while k-step ks multiplies
                if (ks + 1 < KSUB) fread(s, ks + 1, fa[cur ^ 1], fb[cur ^ 1]);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        acc[nt][mt] = mfma32x32x16(fa[cur][nt], fb[cur][mt], acc[nt][mt]);
            }
            // issue order of this step: fragment reads of k-step 0, the global
            // loads of step kt+1, then each k-step's MFMAs interleaved one to
            // one with the next k-step's fragment reads, then the LDS stores
            __builtin_amdgcn_sched_group_barrier(0x100, NT + MT, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, C::A_LOADS + C::B_LOADS, 0);
#pragma unroll
            for (int ks = 0; ks < KSUB - 1; ++ks) {
#pragma unroll
                for (int i = 0; i < NT + MT; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, NT * MT - (NT + MT), 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, NT * MT, 0);
            lstore(buf ^ 1);
            __syncthreads();
        }

        // epilogue: lane holds, per 32x32 tile, columns (tokens) lane%32 and
        // rows (weight rows) 8q + 4*(lane/32) + i for q, i < 4
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int mloc = wm * MT * 32 + mt * 32 + (lane & 31);
            if (mloc >= Mp) continue;
            const int64_t rrow = row0 + m0 + mloc;
            if (UP) {
                constexpr int H = NT / 2;
                bf16_t* hrow = p.h_out + rrow * p.N + nb * C::NOUT + wn * H * 32 + 4 * (lane >> 5);
#pragma unroll
                for (int j = 0; j < H; ++j) {
                    const floatx16& u = acc[j][mt];
                    const floatx16& v = acc[j + H][mt];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        uint2 pk;
                        pk.x = pack_bf16x2(silu(u[4 * q + 0]) * v[4 * q + 0],
                                           silu(u[4 * q + 1]) * v[4 * q + 1]);
                        pk.y = pack_bf16x2(silu(u[4 * q + 2]) * v[4 * q + 2],
                                           silu(u[4 * q + 3]) * v[4 * q + 3]);
                        *reinterpret_cast<uint2*>(hrow + j * 32 + 8 * q) = pk;
                    }
                }
            } else {
                int64_t orow = rrow;
                float gw = 1.0f;
                if (p.topk_w && p.perm) {
                    orow = p.perm[rrow];
                    gw = p.topk_w[orow];
                }
                float* yrow = p.y_out + orow * p.N + nb * C::NOUT + wn * NT * 32 + 4 * (lane >> 5);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        float4 v;
                        v.x = gw * acc[nt][mt][4 * q + 0];
                        v.y = gw * acc[nt][mt][4 * q + 1];
                        v.z = gw * acc[nt][mt][4 * q + 2];
                        v.w = gw * acc[nt][mt][4 * q + 3];
                        *reinterpret_cast<float4*>(yrow + nt * 32 + 8 * q) = v;
                    }
                }
            }
        }
    }
}

int cu_count()
{
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

template <bool UP, int WAVES_N, int WAVES_M, int NT, int MT>
hipError_t run_tiled(const TiledParams& p, int64_t A, hipStream_t stream)
{
    using C = TiledCfg<UP, WAVES_N, WAVES_M, NT, MT>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&tiled_kernel<UP, WAVES_N, WAVES_M, NT, MT>),
            hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    // items are at most nbn * (A/BM + E); never more workgroups than items
    const int64_t nbn = p.N / C::NOUT;
    const int64_t items = nbn * (A / C::BM + p.E);
    int64_t grid = cu_count();
    if (grid > items) grid = items;
    grid = ((grid + 7) / 8) * 8;
    tiled_kernel<UP, WAVES_N, WAVES_M, NT, MT>
        <<<static_cast<unsigned>(grid), C::THREADS, C::LDS_BYTES, stream>>>(p);
    return hipGetLastError();
}

#define MOE_TILED_UP_CFG 4, 2, 2, 4
#define MOE_TILED_DOWN_CFG 4, 2, 2, 4
// UP: 8 waves as 4 (weight rows) x 2 (tokens); 128 w1 + 128 w3 rows x 256 tokens
using UpTile = TiledCfg<true, MOE_TILED_UP_CFG>;
// DOWN: 8 waves as 4 x 2; 256 w2 rows x 256 tokens
using DownTile = TiledCfg<false, MOE_TILED_DOWN_CFG>;

}  // namespace

bool tiled_supported(int d, int ffn)
{
    return ffn % UpTile::NOUT == 0 && d % DownTile::NOUT == 0 && d % 64 == 0 && ffn % 64 == 0;
}

hipError_t launch_tiled_up(const UpArgs& a, hipStream_t stream)
{
    TiledParams p{};
    p.act = a.x;
    p.gather = a.gather;
    p.kslots = a.kslots;
    p.offsets = a.offsets;
    p.wa = a.w1;
    p.wb = a.w3;
    p.N = a.ffn;
    p.K = a.d;
    p.E = a.E;
    p.h_out = a.h;
    return run_tiled<true, MOE_TILED_UP_CFG>(p, a.A, stream);
}

hipError_t launch_tiled_down(const DownArgs& a, hipStream_t stream)
{
    TiledParams p{};
    p.act = a.h;
    p.offsets = a.offsets;
    p.wa = a.w2;
    p.N = a.d;
    p.K = a.ffn;
    p.E = a.E;
    p.y_out = a.y;
    p.topk_w = a.topk_w;
    p.perm = a.perm;
    return run_tiled<false, MOE_TILED_DOWN_CFG>(p, a.A, stream);
}

}  // namespace moe
