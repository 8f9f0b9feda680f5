// Weight-streaming grouped expert GEMMs for decode shapes (few rows per
// expert), gfx950.
//
// In a decode step each active expert sees only a handful of token rows, so
// the layer is bound by reading the expert weights from HBM (arithmetic
// intensity = rows per expert flop/byte, far below the MFMA/HBM ridge).  The
// kernels therefore read every weight byte exactly once:
//
//   * a workgroup owns one expert e and a slab of weight rows; each wave owns
//     16 rows (of w1 or w3 in UP, of w2 in DOWN) and a 1/KS share of the
//     reduction dimension;
//   * weights go straight from HBM into registers as the A operand of a
//     16x16x32 bf16 MFMA (lane l reads 16 contiguous bytes of row l%16), one
//     or two chunks of KC reduction elements ahead of the MFMAs that consume
//     them (two or three register sets); 8-bit weights (E4M3 bytes, one f32
//     scale per row) are widened to bf16 in registers and scaled in the
//     epilogue;
//   * the expert's token rows (<= 16*G per pass) are staged through LDS once
//     per chunk and shared by the NS waves of a reduction share (B operand);
//   * UP pairs waves: one streams 16 rows of w1, its partner the same rows of
//     w3, both against the same token fragments; the partner hands its result
//     over through LDS for the fused SiLU*mul epilogue (h in bf16).  DOWN
//     fuses the gate-weighted scatter of each row back to its (token, slot)
//     position in f32;
//   * partial sums of the KS reduction shares are added in LDS in a fixed
//     order, so results are bitwise reproducible.
//
// Per-expert row counts come from the device-side offsets; experts with no
// rows exit at once and no host synchronisation is needed.  Up to 1024
// assignments a workgroup keeps the routing in LDS: the offsets and the row
// order are read in one round trip, or built from the top-k ids (counts by
// LDS atomics, each row's place by wave ballots, the stable expert-major
// order of the dispatch), so that a decode step needs no dispatch kernel.  An
// expert with more than 16*G rows is cut into several passes over its slab,
// which run as separate workgroups placed to share the slab's weights through
// L2.  With null offsets and no ids the kernels take one matrix of all rows (a
// dense projection).
#include "common.hpp"
#include "launch.hpp"

namespace moe {

namespace {

// assignments (tokens x k) up to which the routing tables live in LDS
constexpr int kListMax = kStreamListMax;

struct StreamParams {
    const bf16_t* act;       // token rows (UP: x, DOWN: h)
    const int32_t* gather;   // UP: source row = gather[r] / kslots (null = r)
    int kslots;
    const int32_t* offsets;  // [E+1]
    const bf16_t* wa;        // UP: w1, DOWN: w2   [E, N, K]
    const bf16_t* wb;        // UP: w3             [E, N, K]
    const uint8_t* qa;       // 8-bit kernels: E4M3 bytes of wa / wb, [E, N, K]
    const uint8_t* qb;
    const float* sa;         // 8-bit kernels: per-row scales of qa / qb, [E, N]
    const float* sb;
    int N, K;                // weight rows / reduction length per expert
    int E;
    bf16_t* h_out;           // UP   [A, N]
    float* y_out;            // DOWN [A, N]
    const float* topk_w;     // DOWN, null = unweighted row order
    const int32_t* perm;     // DOWN
    int passes;              // workgroups per slab (each takes every passes-th pass)
    int mlo, mhi;            // experts with mlo <= rows <= mhi only
    int rows;                // dense (offsets null): one matrix, rows [0, rows)
    // top-k expert of each assignment [A] (A <= kListMax): the row offsets
    // and the expert-major row order are built in LDS from them, and
    // offsets / gather / perm are not read
    const int32_t* ids;
    int A;                   // assignments (rows of all experts)
};

// rows of expert e and its first row (dense: one matrix holding every row)
__device__ __forceinline__ int expert_rows(const StreamParams& p, int e)
{
    return p.offsets ? p.offsets[e + 1] - p.offsets[e] : (e == 0 ? p.rows : 0);
}
__device__ __forceinline__ int expert_row0(const StreamParams& p, int e)
{
    return p.offsets ? p.offsets[e] : 0;
}

// SPLIT (UP only): waves ns < NS/2 stream w1 rows, waves ns >= NS/2 the same
// rows of w3; u and v meet in LDS for the SiLU*mul epilogue.  Each wave then
// carries one matrix, like DOWN, which halves its registers.
template <bool UP, int NS, int KS, int G, int KC, bool SPLIT = false>
struct StreamCfg {
    static constexpr int THREADS = 64 * NS * KS;
    static constexpr int ROWS = SPLIT ? 16 * NS / 2 : 16 * NS;  // output rows per workgroup
    static constexpr int MT = 16 * G;             // token rows per pass (at most)
    static constexpr int LDK = KC + 8;            // padded LDS row (bf16 elements)
    static constexpr int NMAT = (UP && !SPLIT) ? 2 : 1;
    static constexpr int TILE_BYTES = 2 * KS * MT * LDK * 2;  // double-buffered
    static constexpr int RED_BYTES = (KS - 1) * NS * 64 * G * 4 * NMAT * 4;
    static constexpr int SPLIT_BYTES = SPLIT ? (NS / 2) * 64 * G * 4 * 4 : 0;
    static constexpr int LDS_A = TILE_BYTES > RED_BYTES ? TILE_BYTES : RED_BYTES;
    static constexpr int LDS_BYTES = LDS_A > SPLIT_BYTES ? LDS_A : SPLIT_BYTES;
    static_assert(!SPLIT || (UP && KS == 1 && NS % 2 == 0), "SPLIT: UP, no K split, even NS");
};

// Weight registers of one reduction chunk: the raw 16-byte loads that are
// the A operands of KC/32 MFMA k-steps, one load per k-step in bf16, one per
// two k-steps in E4M3.
template <int NLOAD, bool TWO>
struct ChunkRegs {
    uint4 a[NLOAD];
    uint4 b[TWO ? NLOAD : 1];
};

struct PassCtx {
    int e, n0, row0, m0, Mp, ks, ns, gt, lane, kbeg, nchunks, rot;
    // the assignment behind each expert-major row, in LDS (null: read perm /
    // gather from global memory); gather: UP rows come from x[assignment / k];
    // scatter: DOWN rows go to y[assignment], gate-weighted
    const int* list;
    bool gather, scatter;
    const bf16_t* pa;
    const bf16_t* pb;
    const uint8_t* qa;  // 8-bit kernels: this lane's weight bytes
    const uint8_t* qb;
    const float* sa;    // 8-bit kernels: scales of this wave's weight rows
    const float* sb;
};

// One pass over at most 16*GA token rows of expert e for this workgroup's
// weight rows.  GA is the number of 16-row groups actually computed (a
// compile-time count, so the MFMA sequence has no data-dependent branches).
// F8: the weights are E4M3 bytes with per-row scales.  A 16-byte load then
// holds 16 consecutive reduction elements of a row, which feed two k-steps;
// the reduction order is permuted accordingly (lane l, k-step 2j + h takes
// elements 64j + 16 (l / 16) + 8h .. +7) and the token fragments are read in
// the same order.  The row scales multiply the accumulators.
// ST weight register sets: chunk c is multiplied while the weights of chunks
// c+1 .. c+ST-1 are in flight (the token tile is always one chunk ahead).
template <bool UP, int NS, int KS, int G, int KC, int GA, bool SPLIT, bool F8, int ST>
__device__ __forceinline__ void stream_pass(const StreamParams& p, unsigned char* smem,
                                            const PassCtx& x)
{
    using C = StreamCfg<UP, NS, KS, G, KC, SPLIT>;
    constexpr bool TWO = UP && !SPLIT;  // two weight matrices per wave
    constexpr int KSTEPS = KC / 32;
    constexpr int NLOAD = F8 ? KSTEPS / 2 : KSTEPS;
    static_assert(!F8 || KC % 64 == 0, "E4M3 chunks hold whole 64-element row segments");
    static_assert(ST == 2 || ST == 3, "two or three weight register sets");
    constexpr int GT = 64 * NS;  // threads that stage one token tile
    constexpr int TILE_LOADS = 16 * GA * KC / 8;
    constexpr int TPT = (TILE_LOADS + GT - 1) / GT;
    // two token tiles per reduction share, used by alternate chunks
    bf16_t* tiles = reinterpret_cast<bf16_t*>(smem) + x.ks * 2 * C::MT * C::LDK;
    const int lane = x.lane;

    const bf16_t* src[TPT];
    int ldsoff[TPT];
#pragma unroll
    for (int it = 0; it < TPT; ++it) {
        const int q = it * GT + x.gt;
        const bool live = (TILE_LOADS % GT == 0) || q < TILE_LOADS;
        const int m = live ? q / (KC / 8) : 0;
        const int c8 = live ? q % (KC / 8) : 0;
        const int mm = m < x.Mp ? m : x.Mp - 1;  // rows past the end repeat the last row
        const int r = x.row0 + x.m0 + mm;
        int64_t sr = r;
        if (UP && x.gather) sr = (x.list ? x.list[r] : p.gather[r]) / p.kslots;
        src[it] = p.act + sr * p.K + x.kbeg + c8 * 8;
        ldsoff[it] = live ? m * C::LDK + c8 * 8 : -1;
    }

    floatx4 accA[GA], accB[GA];
#pragma unroll
    for (int g = 0; g < GA; ++g) {
        accA[g] = floatx4{0.f, 0.f, 0.f, 0.f};
        accB[g] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

    using R = ChunkRegs<NLOAD, TWO>;
    uint4 tok[TPT];
    // chunk c starts at column (c + rot) mod nchunks of the slab; c is clamped
    // to the last chunk, whose loads then repeat (see step)
    auto kofs = [&](int c) {
        c = c < x.nchunks ? c : x.nchunks - 1;
        const int cr = c + x.rot;
        return (cr < x.nchunks ? cr : cr - x.nchunks) * KC;
    };
    auto load_t = [&](int c) {
        const int ko = kofs(c);
#pragma unroll
        for (int it = 0; it < TPT; ++it)
            if (ldsoff[it] >= 0) tok[it] = ldg16(src[it] + ko);
    };
    auto load_w = [&](R& r, int c) {
        const int ko = kofs(c);
#pragma unroll
        for (int j = 0; j < NLOAD; ++j) {
            if constexpr (F8) {
                r.a[j] = ldg16(x.qa + ko + j * 64);
                if (TWO) r.b[j] = ldg16(x.qb + ko + j * 64);
            } else {
                r.a[j] = ldg16(x.pa + ko + j * 32);
                if (TWO) r.b[j] = ldg16(x.pb + ko + j * 32);
            }
        }
    };
    // the A operand of k-step kk
    auto opnd = [](const uint4* w, int kk) -> bf16x8 {
        if constexpr (F8) {
            const uint4 v = w[kk >> 1];
            return (kk & 1) ? e4m3x8_to_bf16(v.z, v.w) : e4m3x8_to_bf16(v.x, v.y);
        } else {
            return as_bf16x8(w[kk]);
        }
    };
    // Stage chunk c's tokens, load chunk c+1's tokens and chunk c+ST-1's
    // weights (into the set chunk c-1 used), multiply chunk c.  The loads are
    // unconditional (past the last chunk they repeat it) so that the
    // compiler's memory-counter waits stay exact; they retire in issue order,
    // so waiting for chunk c's tokens (issued after chunk c's weights and
    // before chunk c+1's) leaves chunks c+1 .. c+ST-1 in flight.  Chunk c's
    // tile is the one chunk c-2 read; every wave finished those reads before
    // it reached chunk c-1's barrier, so one barrier per chunk suffices.
    auto step = [&](int c, R& cur, R& ahead) {
        bf16_t* tile = tiles + (c & 1) * C::MT * C::LDK;
#pragma unroll
        for (int it = 0; it < TPT; ++it)
            if (ldsoff[it] >= 0) *reinterpret_cast<uint4*>(tile + ldsoff[it]) = tok[it];
        load_t(c + 1);
        load_w(ahead, c + ST - 1);
        // E4M3: keep the first conversion (which waits for this chunk's
        // weights) below the new loads, or fewer chunks would be in flight
        if constexpr (F8) __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) {
            const bf16x8 a = opnd(cur.a, kk);
            const bf16x8 a2 = TWO ? opnd(cur.b, kk) : a;
            const int kcol = F8 ? (kk >> 1) * 64 + 16 * (lane >> 4) + 8 * (kk & 1)
                                : kk * 32 + 8 * (lane >> 4);
#pragma unroll
            for (int g = 0; g < GA; ++g) {
                const bf16x8 b = *reinterpret_cast<const bf16x8*>(
                    tile + (g * 16 + (lane & 15)) * C::LDK + kcol);
                accA[g] = mfma16x16x32(a, b, accA[g]);
                if (TWO) accB[g] = mfma16x16x32(a2, b, accB[g]);
            }
        }
    };

    R r0, r1, r2;
    load_t(0);
    load_w(r0, 0);
    if constexpr (ST == 3) load_w(r1, 1);
    __syncthreads();  // the previous pass (or reduction) is done with the LDS
    if constexpr (ST == 2) {
        for (int c = 0; c < x.nchunks; c += 2) {
            step(c, r0, r1);
            if (c + 1 < x.nchunks) step(c + 1, r1, r0);
        }
    } else {
        for (int c = 0; c < x.nchunks; c += 3) {
            step(c, r0, r2);
            if (c + 1 < x.nchunks) step(c + 1, r1, r0);
            if (c + 2 < x.nchunks) step(c + 2, r2, r1);
        }
    }

    if (KS > 1) {
        // add the reduction shares ks = 1..KS-1 into share 0, in order
        __syncthreads();
        float* red = reinterpret_cast<float*>(smem);
        constexpr int SLOT = 64 * G * 4 * C::NMAT;
        if (x.ks > 0) {
            float* dst = red + ((x.ks - 1) * NS + x.ns) * SLOT;
#pragma unroll
            for (int g = 0; g < GA; ++g) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    dst[((g * 4 + i) * C::NMAT + 0) * 64 + lane] = accA[g][i];
                    if (UP) dst[((g * 4 + i) * C::NMAT + 1) * 64 + lane] = accB[g][i];
                }
            }
        }
        __syncthreads();
        if (x.ks == 0) {
            for (int s = 1; s < KS; ++s) {
                const float* sr = red + ((s - 1) * NS + x.ns) * SLOT;
#pragma unroll
                for (int g = 0; g < GA; ++g) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        accA[g][i] += sr[((g * 4 + i) * C::NMAT + 0) * 64 + lane];
                        if (UP) accB[g][i] += sr[((g * 4 + i) * C::NMAT + 1) * 64 + lane];
                    }
                }
            }
        }
    }

    if constexpr (F8) {
        // row scales: lane holds output rows n0 + 4 (lane / 16) + i
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float s1 = x.sa[4 * (lane >> 4) + i];
            const float s2 = TWO ? x.sb[4 * (lane >> 4) + i] : 0.0f;
#pragma unroll
            for (int g = 0; g < GA; ++g) {
                accA[g][i] *= s1;
                if (TWO) accB[g][i] *= s2;
            }
        }
    }

    if constexpr (SPLIT) {
        // the w3 waves hand v to the w1 waves of the same output rows
        __syncthreads();
        float* xv = reinterpret_cast<float*>(smem);
        const int pair = x.ns % (NS / 2);
        if (x.ns >= NS / 2) {
#pragma unroll
            for (int g = 0; g < GA; ++g)
#pragma unroll
                for (int i = 0; i < 4; ++i) xv[((pair * G + g) * 4 + i) * 64 + lane] = accA[g][i];
        }
        __syncthreads();
        if (x.ns < NS / 2) {
#pragma unroll
            for (int g = 0; g < GA; ++g)
#pragma unroll
                for (int i = 0; i < 4; ++i) accB[g][i] = xv[((pair * G + g) * 4 + i) * 64 + lane];
        }
    }

    if (x.ks == 0 && (!SPLIT || x.ns < NS / 2)) {
        const int n = x.n0 + 4 * (lane >> 4);
#pragma unroll
        for (int g = 0; g < GA; ++g) {
            const int tok = g * 16 + (lane & 15);
            if (tok < x.Mp) {
                const int64_t r = x.row0 + x.m0 + tok;
                if (UP) {
                    uint2 pk;
                    pk.x = pack_bf16x2(silu(accA[g][0]) * accB[g][0], silu(accA[g][1]) * accB[g][1]);
                    pk.y = pack_bf16x2(silu(accA[g][2]) * accB[g][2], silu(accA[g][3]) * accB[g][3]);
                    *reinterpret_cast<uint2*>(p.h_out + r * p.N + n) = pk;
                } else {
                    int64_t orow = r;
                    float gw = 1.0f;
                    if (x.scatter) {
                        orow = x.list ? x.list[r] : p.perm[r];
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
    // the LDS tile/reduction area is reused by the next pass
    __syncthreads();
}

template <bool UP, int NS, int KS, int G, int KC, bool SPLIT, bool F8, int ST>
__global__ __launch_bounds__(64 * NS * KS) void stream_kernel(StreamParams p)
{
    using C = StreamCfg<UP, NS, KS, G, KC, SPLIT>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::LDS_BYTES];

    // Workgroup -> (expert e, slab nb, pass slot q).  An expert's rows are
    // cut into P_e = ceil(M_e/MT) balanced passes and it gets Q_e =
    // min(P_e, passes) pass slots per slab; slot q takes passes q, q + Q_e, ...
    // The items are numbered densely, expert-major, and within an expert
    // (group of 8 slabs, pass slot, slab % 8).  Dispatch places workgroup b
    // on XCD b % 8.  UP takes item b: the 8 slabs of a group run on the 8
    // XCDs, and all pass slots of a slab land on one XCD one after another,
    // re-reading the slab's weights from its L2.  DOWN cuts the list into 8
    // contiguous ranges, one per XCD: its token rows (h, ffn values each) of
    // all experts overflow an L2 while those of one or two experts fit, and
    // every slab re-reads them (measured 10-28% faster at 45-64 rows per
    // expert).  UP's token rows are 3.5x shorter and fit anyway, and there
    // the ranges would crowd a heavy expert's MFMA-bound passes onto one or
    // two XCDs.  The workgroups past the last item (the grid is sized for the
    // worst case) exit at once.
    __shared__ int s_first[65];  // first item of expert e
    // Routing tables in LDS, for up to kListMax assignments: the expert row
    // offsets and the assignment behind each expert-major row.  Loaded
    // together (one memory round trip where the offsets and then the row
    // order would take two), or built here from the top-k ids, which spares
    // the step a separate dispatch kernel.
    __shared__ int s_off[65];
    __shared__ int s_list[kListMax];
    __shared__ int s_wc[C::THREADS / 64];
    constexpr int IPT = (kListMax + C::THREADS - 1) / C::THREADS;  // ids per thread
    const int nbn = p.N / C::ROWS;
    const int nbn8 = (nbn + 7) & ~7;
    const int tid = threadIdx.x;
    const bool by_ids = p.ids != nullptr;
    const bool tab = by_ids || (p.offsets && p.A <= kListMax);
    // UP: the gather source of each row; DOWN: the scatter target
    const int32_t* const rperm = UP ? p.gather : ((p.topk_w && p.perm) ? p.perm : nullptr);
    int myid[IPT];
    if (by_ids) {
        // s_off counts first, then holds the offsets
        if (tid < 64) s_off[tid] = 0;
#pragma unroll
        for (int i = 0; i < IPT; ++i) {
            const int a = i * C::THREADS + tid;
            // ids come from the router and lie in [0, E); the clamp keeps a
            // corrupted id from indexing past the counts
            myid[i] = a < p.A ? min(max(p.ids[a], 0), p.E - 1) : -1;
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < IPT; ++i)
            if (myid[i] >= 0) atomicAdd(&s_off[myid[i]], 1);
        __syncthreads();
    } else if (tab) {
        if (tid <= p.E) s_off[tid] = p.offsets[tid];
        if (rperm)
            for (int a = tid; a < p.A; a += C::THREADS) s_list[a] = rperm[a];
        __syncthreads();
    }
    if (tid < 64) {
        const int t = tid;
        int Mt = 0;
        if (t < p.E) Mt = by_ids ? s_off[t] : (tab ? s_off[t + 1] - s_off[t] : expert_rows(p, t));
        int items = 0;
        if (t < p.E) {
            const int P = (Mt + C::MT - 1) / C::MT;
            if (Mt >= p.mlo && Mt <= p.mhi) items = nbn8 * (P < p.passes ? P : p.passes);
        }
        // inclusive scans over the wave: items, and (from ids) rows
        int rows = Mt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(items, o, 64);
            const int w = __shfl_up(rows, o, 64);
            if (t >= o) {
                items += v;
                rows += w;
            }
        }
        if (t < p.E) s_first[t + 1] = items;
        if (t == 0) s_first[0] = 0;
        if (by_ids) {
            if (t < p.E) s_off[t] = rows - Mt;
            if (t == p.E - 1) s_off[p.E] = rows;
        }
    }
    __syncthreads();
    const int total = s_first[p.E];
    int b = static_cast<int>(blockIdx.x);
    if constexpr (UP) {
        if (b >= total) return;
    } else {
        const int per_xcd = (total + 7) >> 3;
        const int j = b >> 3;
        b = (b & 7) * per_xcd + j;
        if (j >= per_xcd || b >= total) return;
    }
    int e = 0;
    while (s_first[e + 1] <= b) ++e;
    const int row0 = tab ? s_off[e] : expert_row0(p, e);
    const int M = tab ? s_off[e + 1] - s_off[e] : expert_rows(p, e);
    const int npass = (M + C::MT - 1) / C::MT;
    const int nslot = npass < p.passes ? npass : p.passes;
    const int local = b - s_first[e];
    const int grp = local / (8 * nslot);
    const int rem = local - grp * 8 * nslot;
    const int q = rem >> 3;
    const int nb = grp * 8 + (rem & 7);
    if (nb >= nbn) return;
    const int rp = (M + npass - 1) / npass;  // rows per pass, balanced

    PassCtx x;
    x.gather = UP && (by_ids || p.gather);
    x.scatter = !UP && p.topk_w && (by_ids || p.perm);
    x.list = tab ? s_list : nullptr;
    if (by_ids && (x.gather || x.scatter)) {
        // this expert's rows in assignment order (stable): a wave ballot and
        // the counts of the waves before give each of its assignments a row
        const int lane = tid & 63, wv = tid >> 6;
        const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
        int base = row0;
#pragma unroll
        for (int i = 0; i < IPT; ++i) {
            if (i * C::THREADS < p.A) {
                const bool mine = myid[i] == e;
                const uint64_t bal = __ballot(mine);
                if (lane == 0) s_wc[wv] = __popcll(bal);
                __syncthreads();
                int before = 0, tot = 0;
#pragma unroll
                for (int w = 0; w < C::THREADS / 64; ++w) {
                    const int c = s_wc[w];
                    tot += c;
                    before += w < wv ? c : 0;
                }
                if (mine) s_list[base + before + __popcll(bal & lt)] = i * C::THREADS + tid;
                base += tot;
                __syncthreads();
            }
        }
    }
    x.lane = tid & 63;
    const int wave = tid >> 6;
    x.ns = wave % NS;
    x.ks = wave / NS;
    x.gt = tid % (64 * NS);
    x.e = e;
    x.n0 = nb * C::ROWS + (SPLIT ? x.ns % (NS / 2) : x.ns) * 16;
    x.row0 = row0;
    const int kper = p.K / KS;
    x.kbeg = x.ks * kper;
    x.nchunks = kper / KC;
    // Each slab walks its chunks starting at a rotated position, so the
    // workgroups in flight read different columns of their rows at any one
    // time (all starting at column 0 measured about 10% slower).  Slabs of one
    // group of 8 (one per XCD) share a rotation, and so do the passes of a
    // slab, which then read the same chunks at about the same time.  The
    // reduction order changes with it; results stay deterministic.
    x.rot = static_cast<int>((static_cast<unsigned>(e * (nbn8 >> 3) + grp) * 5u) %
                             static_cast<unsigned>(x.nchunks));
    const int64_t wrow = (int64_t)e * p.N + x.n0 + (x.lane & 15);
    const int64_t srow = (int64_t)e * p.N + x.n0;  // first row of this wave's 16
    if constexpr (F8) {
        const bool w3 = SPLIT && x.ns >= NS / 2;
        x.qa = (w3 ? p.qb : p.qa) + wrow * p.K + x.kbeg + 16 * (x.lane >> 4);
        x.qb = (UP && !SPLIT) ? p.qb + wrow * p.K + x.kbeg + 16 * (x.lane >> 4) : nullptr;
        x.sa = (w3 ? p.sb : p.sa) + srow;
        x.sb = (UP && !SPLIT) ? p.sb + srow : nullptr;
        x.pa = x.pb = nullptr;
    } else if (SPLIT) {
        x.pa = (x.ns < NS / 2 ? p.wa : p.wb) + wrow * p.K + x.kbeg + 8 * (x.lane >> 4);
        x.pb = nullptr;
    } else {
        x.pa = p.wa + wrow * p.K + x.kbeg + 8 * (x.lane >> 4);
        x.pb = UP ? p.wb + wrow * p.K + x.kbeg + 8 * (x.lane >> 4) : nullptr;
    }

    for (int pass = q; pass < npass; pass += nslot) {
        x.m0 = pass * rp;
        x.Mp = min(M - x.m0, rp);
        // the pass multiplies exactly the 16-row groups that hold rows (a
        // 45-row pass: 3 groups, not 4; measured 3-7% faster at 45-97 rows)
        const int gact = (x.Mp + 15) >> 4;
        switch (gact) {
        case 1: stream_pass<UP, NS, KS, G, KC, 1, SPLIT, F8, ST>(p, smem, x); break;
        case 2: if constexpr (G >= 2) stream_pass<UP, NS, KS, G, KC, 2, SPLIT, F8, ST>(p, smem, x); break;
        case 3: if constexpr (G >= 3) stream_pass<UP, NS, KS, G, KC, 3, SPLIT, F8, ST>(p, smem, x); break;
        case 4: if constexpr (G >= 4) stream_pass<UP, NS, KS, G, KC, 4, SPLIT, F8, ST>(p, smem, x); break;
        case 5: if constexpr (G >= 5) stream_pass<UP, NS, KS, G, KC, 5, SPLIT, F8, ST>(p, smem, x); break;
        case 6: if constexpr (G >= 6) stream_pass<UP, NS, KS, G, KC, 6, SPLIT, F8, ST>(p, smem, x); break;
        case 7: if constexpr (G >= 7) stream_pass<UP, NS, KS, G, KC, 7, SPLIT, F8, ST>(p, smem, x); break;
        case 8: if constexpr (G >= 8) stream_pass<UP, NS, KS, G, KC, 8, SPLIT, F8, ST>(p, smem, x); break;
        default: if constexpr (G >= 16) stream_pass<UP, NS, KS, G, KC, 16, SPLIT, F8, ST>(p, smem, x); break;
        }
    }
}

template <bool UP, int NS, int KS, int G, int KC, bool SPLIT = false, bool F8 = false, int ST = 2>
hipError_t run(StreamParams p, int64_t rows_max, hipStream_t stream)
{
    // pass slots per slab: enough for an expert that takes rows_max rows
    // (every token at most once), at most 8
    constexpr int MT = StreamCfg<UP, NS, KS, G, KC, SPLIT>::MT;
    const int64_t need = (rows_max + MT - 1) / MT;
    p.passes = static_cast<int>(need < 1 ? 1 : (need > 8 ? 8 : need));
    using C = StreamCfg<UP, NS, KS, G, KC, SPLIT>;
    const int nbn8 = (p.N / C::ROWS + 7) & ~7;
    const unsigned grid = static_cast<unsigned>(p.E * nbn8 * p.passes);
    stream_kernel<UP, NS, KS, G, KC, SPLIT, F8, ST><<<grid, C::THREADS, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace

// Tile shape by the mean rows per expert (A/E), from sweeps on MI355X at the
// Mixtral shapes: 32-row passes while the mean is small, 64-row passes above
// (128-row passes for the up GEMM above a mean of 48); an expert with more
// rows than one pass holds is cut into several passes, which run as separate
// workgroups.  The chunk length KC trades bytes in flight against registers.
int stream_groups(int64_t A, int E, int64_t rows_max)
{
    const int64_t mean = (A + E - 1) / E;
    const int g = mean <= 24 ? 2 : (mean <= 48 ? 4 : 8);
    // no expert has more than rows_max rows: 64-row passes hold any of them
    return (g > 4 && rows_max <= 64) ? 4 : g;
}

hipError_t launch_stream_up(const UpArgs& a, int64_t rows_max, hipStream_t stream)
{
    StreamParams p{};
    p.act = a.x;
    p.gather = a.gather;
    p.kslots = a.kslots;
    p.ids = a.ids;
    p.A = static_cast<int>(a.A < 0x7fffffff ? a.A : 0x7fffffff);
    if (a.ids && a.A > kListMax) return hipErrorInvalidValue;
    p.offsets = a.offsets;
    p.wa = a.w1;
    p.wb = a.w3;
    p.qa = a.q1;
    p.qb = a.q3;
    p.sa = a.s1;
    p.sb = a.s3;
    p.N = a.ffn;
    p.K = a.d;
    p.E = a.E;
    p.h_out = a.h;
    p.mlo = a.mlo;
    p.mhi = a.mhi;
    const int G = a.groups ? a.groups : stream_groups(a.A, a.E, rows_max);
    // 8 waves: 4 stream w1 rows, 4 the same w3 rows (SPLIT)
    if (a.q1) {
        // E4M3 (sweeps on MI355X): 256-element chunks for up to 32 rows per
        // pass; 512 would hold the bf16 kernel's bytes in flight but needs
        // 154 VGPRs, one workgroup per CU, and measured 13% slower
        if (G == 2) {
            if (a.d % 256 == 0) return run<true, 8, 1, 2, 256, true, true>(p, rows_max, stream);
            if (a.d % 128 == 0) return run<true, 8, 1, 2, 128, true, true>(p, rows_max, stream);
            return run<true, 8, 1, 2, 64, true, true>(p, rows_max, stream);
        }
        if (G == 8) {
            if (a.d % 128 == 0) return run<true, 8, 1, 8, 128, true, true>(p, rows_max, stream);
            return run<true, 8, 1, 8, 64, true, true>(p, rows_max, stream);
        }
        if (a.d % 128 == 0) return run<true, 8, 1, 4, 128, true, true>(p, rows_max, stream);
        return run<true, 8, 1, 4, 64, true, true>(p, rows_max, stream);
    }
    if (G == 2) {
        if (a.d % 256 == 0) return run<true, 8, 1, 2, 256, true>(p, rows_max, stream);
        if (a.d % 128 == 0) return run<true, 8, 1, 2, 128, true>(p, rows_max, stream);
        return run<true, 8, 1, 2, 64, true>(p, rows_max, stream);
    }
    if (G == 8) return run<true, 8, 1, 8, 64, true>(p, rows_max, stream);
    if (a.d % 128 == 0) return run<true, 8, 1, 4, 128, true>(p, rows_max, stream);
    return run<true, 8, 1, 4, 64, true>(p, rows_max, stream);
}

hipError_t launch_stream_down(const DownArgs& a, int64_t rows_max, hipStream_t stream)
{
    StreamParams p{};
    p.act = a.h;
    p.offsets = a.offsets;
    p.wa = a.w2;
    p.qa = a.q2;
    p.sa = a.s2;
    p.N = a.d;
    p.K = a.ffn;
    p.E = a.E;
    p.y_out = a.y;
    p.topk_w = a.topk_w;
    p.perm = a.perm;
    p.ids = a.ids;
    p.A = static_cast<int>(a.A < 0x7fffffff ? a.A : 0x7fffffff);
    if (a.ids && a.A > kListMax) return hipErrorInvalidValue;
    p.mlo = a.mlo;
    p.mhi = a.mhi;
    p.rows = static_cast<int>(a.A);
    const int G = a.groups ? a.groups : stream_groups(a.A, a.E, rows_max);
    if (!a.offsets && !a.ids) {
        // the dense shapes below exist for bf16 weights only
        if (a.q2) return hipErrorInvalidValue;
        // dense projection (one matrix): several reduction shares per
        // workgroup, so that a single matrix still spreads over the CUs.
        // Measured on MI355X, K = 4096: more than 4096 output rows, 2 row
        // waves x 4 shares with 64-token passes (6144 rows: 23 -> 18 us at 64
        // tokens, 19 -> 12 us at 8); up to 24 tokens, 16-row slabs (4096 rows
        // at 8 tokens: 11.6 -> 8.3 us); otherwise 2 row waves x 4 shares
        // with 32-token passes (2 workgroups per slab, the second re-reading
        // it from L2; 4096 rows at 64 tokens: 23 -> 14 us)
        if (a.ffn % 512 == 0) {
            if (a.d > 4096) return run<false, 2, 4, 4, 128>(p, rows_max, stream);
            if (G == 2) return run<false, 1, 4, 2, 128>(p, rows_max, stream);
            return run<false, 2, 4, 2, 128>(p, rows_max, stream);
        }
        if (a.ffn % 256 == 0) {
            if (G == 2) return run<false, 4, 4, 2, 64>(p, rows_max, stream);
            return run<false, 4, 4, 4, 64>(p, rows_max, stream);
        }
        return run<false, 4, 1, 4, 64>(p, rows_max, stream);
    }
    if (a.q2) {
        if (G == 2) {
            if (a.d % 128 == 0 && a.ffn % 256 == 0)
                return run<false, 8, 1, 2, 256, false, true>(p, rows_max, stream);
            if (a.d % 128 == 0 && a.ffn % 128 == 0)
                return run<false, 8, 1, 2, 128, false, true>(p, rows_max, stream);
            return run<false, 4, 1, 2, 64, false, true>(p, rows_max, stream);
        }
        if (G == 4 && a.d % 128 == 0 && a.ffn % 128 == 0)
            return run<false, 8, 1, 4, 128, false, true, 3>(p, rows_max, stream);
        if (a.ffn % 128 == 0) return run<false, 4, 1, 4, 128, false, true>(p, rows_max, stream);
        return run<false, 4, 1, 4, 64, false, true>(p, rows_max, stream);
    }
    if (G == 2) {
        if (a.d % 128 == 0 && a.ffn % 128 == 0) return run<false, 8, 1, 2, 128>(p, rows_max, stream);
        return run<false, 4, 1, 2, 64>(p, rows_max, stream);
    }
    // up to 64 rows per pass: 8 waves (128 output rows) share each staged
    // token tile and three weight sets are in flight; above, 4 waves, so a
    // heavy expert's passes spread over twice as many workgroups
    if (G == 4 && a.d % 128 == 0 && a.ffn % 128 == 0)
        return run<false, 8, 1, 4, 128, false, false, 3>(p, rows_max, stream);
    if (a.ffn % 128 == 0) return run<false, 4, 1, 4, 128>(p, rows_max, stream);
    return run<false, 4, 1, 4, 64>(p, rows_max, stream);
}

}  // namespace moe
