// Tiled grouped expert GEMMs for prefill shapes (many rows per expert), gfx950.
//
// With ~1000 token rows per expert the expert FFN is MFMA-bound (arithmetic
// intensity ~ rows per expert flop/byte, above the MI355X ridge of ~310), so
// the kernels reuse both operands from LDS:
//
//   * a workgroup computes a 256 x 256 tile of the output (256 weight rows x
//     256 token rows) with 32x32x16 bf16 MFMAs, f32 accumulation;
//   * UP stages 128 rows of w1 and the same 128 rows of w3, and each wave
//     holds both accumulators of an output element in the same lane, so the
//     SiLU*mul epilogue needs no data movement; token rows are gathered
//     through the dispatch permutation while loading (no separate permute);
//   * DOWN scales each output row by its gate weight and scatters it to the
//     row's (token, slot) position;
//   * workgroups are persistent: one per CU.  The items, ordered expert,
//     weight block, token tile, are cut into 8 contiguous ranges, one per
//     XCD, and the P workgroups of an XCD take the items of its range in
//     turn (workgroup j: items j, j + P, j + 2P, ...), so at any time they
//     work on the token tiles of a few weight blocks and share both operands
//     through that XCD's L2.  Per-expert tile counts are read from the
//     device-side offsets: ragged row counts need no host synchronisation;
//   * DOWN may cut each tile's reduction into parts (a power of two up to
//     the caller's limit; items then ordered expert, part, weight block,
//     token tile), chosen on the device from the tile count by a cost model,
//     where that evens out the rounds of the persistent grid;
//   * or, where the caller's spare slices hold one 256 x 256 f32 piece per
//     workgroup, DOWN leaves the tiles uncut (the tail split): the tiles of
//     the grid's whole rounds, every tile but the experts' short last tiles
//     first, go to the XCDs in equal counts, and each tile left over is cut
//     into contiguous reduction ranges spread over all the workgroups, its
//     pieces added into y by fold_tail_kernel in piece order;
//   * 8-bit weights (E4M3 bytes, one f32 scale per weight row) are staged in
//     LDS as bytes, widened to bf16 at the fragment reads, and their scales
//     multiply the accumulators in the epilogue;
//   * with null offsets the kernel takes one matrix of all rows (a dense
//     projection).
#include <atomic>
#include <mutex>
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace moe {

namespace {

struct TiledParams {
    const bf16_t* act;       // token rows (UP: x, DOWN: h)
    const int32_t* gather;   // UP: source row = gather[r] / kslots (null = r)
    int kslots;
    const int32_t* offsets;  // [E+1]; null: one matrix (E = 1) of all A rows
    const bf16_t* wa;        // UP: w1, DOWN: w2  [E, N, K]
    const bf16_t* wb;        // UP: w3            [E, N, K]
    // 8-bit weights (then wa/wb are unused): E4M3 bytes [E, N, K] and per-row
    // f32 scales [E, N], applied to the accumulators in the epilogue
    const uint8_t* qa;
    const uint8_t* qb;
    const float* sa;
    const float* sb;
    int N, K, E;             // N = weight rows per expert (UP: ffn, DOWN: d)
    bf16_t* h_out;           // UP   [A, N]
    float* y_out;            // DOWN [A, N]
    const float* topk_w;     // DOWN, null = unweighted row order
    const int32_t* perm;     // DOWN
    int mlo, mhi;            // experts with mlo <= rows <= mhi only
    // DOWN: the reduction may be cut into up to ksplit_max parts, part s
    // writing the slice y_out + s * slice; the parts chosen are stored to
    // *ksplit_out (if not null) for the kernel that sums the slices
    int ksplit_max;
    int64_t slice;
    int* ksplit_out;
    int64_t A;
    // DOWN, tail split (see the kernel): tiles uncut, the tiles past the
    // grid's whole rounds split across all the workgroups; the pieces after
    // each tile's first go to y_out + slice (kTailPiece floats each, one slot
    // per workgroup), a table of the split tiles and their count after them
    int tail;
};

// one piece of a split tile: 256 rows x 256 columns of f32
constexpr int kTailPiece = 256 * 256;

int cu_count();

constexpr int kMaxDevices = 64;

// ---- four-wave schedule ------------------------------------------------------
//
// Each tile is computed by 4 waves, one per SIMD, each owning a 128 x 128
// quarter (16 accumulator tiles of 32 x 32, 256 accumulator registers per
// lane).  Measured on MI355X: a wave that interleaves about one 1 KB
// global->LDS load with four 32x32x16 MFMAs keeps the MFMA pipe ~85% busy
// and sustains the 256 x 256 tile's load rate, while loads issued by a second
// wave on a SIMD whose MFMAs run back to back are throttled to about one per
// 32 cycles per CU.  So every wave carries its own loads, fragment reads and
// MFMAs in one interleaved instruction stream (its order pinned with
// scheduling barriers).
//
//   * operands go from global memory straight into LDS (16-byte loads that
//     write LDS at base + 16 * lane, no registers); a step holds BK = 64
//     reduction elements, so one load covers 8 rows x 128 bytes (whole cache
//     lines; half-line rows measured 1.7x slower to issue);
//   * the weight tile A (256 rows) lives in a ring of 3 slots, the token tile
//     B (256 rows) in a ring of 2: 96 + 64 KB, all of the LDS;
//   * step j multiplies its 4 k-steps of 16; while k-step ks multiplies, the
//     fragments of k-step ks+1 are read (in k-step 3: k-step 0 of step j+1),
//     and the wave issues its share of B(j+1) in k-step 0 and of A(j+2) in
//     k-steps 1-2.  After k-step 2 every wave waits for its fragment reads of
//     step j and for its loads up to B(j+1) (loads retire in order), then one
//     barrier makes A(j+1) and B(j+1) complete for all waves and frees the
//     slots of A(j) and B(j) for the next step's loads;
//   * LDS rows are 128 bytes, unpadded; the eight 16-byte chunks of row r are
//     stored at slot chunk ^ ((r >> 1) & 7), so every fragment read (16
//     consecutive rows, one chunk) hits 16 distinct bank groups;
//   * loads past the last step re-load the last step into the free slot, so
//     the wait counts are the same every step.
template <bool UP, bool F8>
struct QCfg {
    static constexpr int THREADS = 256;
    static constexpr int BN = 256;                 // weight rows staged (UP: 128 w1 + 128 w3)
    static constexpr int BM = 256;                 // token rows
    static constexpr int NOUT = UP ? BN / 2 : BN;  // output columns per tile
    static constexpr int BK = 64;
    static constexpr int ROWB = BK * 2;            // bytes per LDS token row
    static constexpr int AROWB = F8 ? BK : BK * 2; // bytes per LDS weight row
    static constexpr int SLOT = 256 * ROWB;        // 32 KB, the token tile of one step
    static constexpr int ASLOT = 256 * AROWB;      // the weight tile of one step (32 or 16 KB)
    static constexpr int B_OFF = 3 * ASLOT;
    static constexpr int LDS_BYTES = 3 * ASLOT + 2 * SLOT;
    static constexpr int NT = 4, MT = 4;           // 32x32 tiles per wave: 128 weight rows x 128 tokens
    static constexpr int LOADS = 8;                // 1 KB token loads per wave per step
    static constexpr int ALOADS = F8 ? 4 : 8;      // 1 KB weight loads per wave per step
};

__device__ __forceinline__ int q_swz(int r) { return (r >> 1) & 7; }

// Relative cost of a tile by the 32-row token blocks each token wave
// multiplies (NMT = ceil(blocks / 2)): a step still loads the whole weight
// tile, so a tile of a few rows costs about half a full one.
constexpr int kFullTileCost = 20;
__device__ __forceinline__ int tile_cost(int rows)
{
    const int nmt = ((rows + 31) / 32 + 1) / 2;
    return nmt >= 4 ? 20 : (nmt == 3 ? 16 : (nmt == 2 ? 12 : 9));
}

// s_waitcnt with only the vector-memory count constrained (expcnt/lgkmcnt at max)
template <int N>
__device__ __forceinline__ void wait_vmem()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | 0xF00 | (((N >> 4) & 3) << 14));
}

// s_waitcnt lgkmcnt(0) with vmcnt/expcnt at max
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time
template <int I, int N, class F>
__device__ __forceinline__ void static_for_from(F&& f)
{
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for_from<I + 1, N>(f);
    }
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f)
{
    static_for_from<0, N>(f);
}

template <bool UP, bool F8>
__global__ __launch_bounds__(256) void q_kernel(TiledParams p)
{
    using C = QCfg<UP, F8>;
    constexpr int NT = C::NT, MT = C::MT, L = C::LOADS, LA = C::ALOADS;
    extern __shared__ __attribute__((aligned(16))) unsigned char ring[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave & 1;   // weight half of this wave
    const int wm = wave >> 1;  // token half of this wave
    const int nbn = p.N / C::NOUT;

    // per-expert token tiles and their prefix, one expert per lane:
    // items before expert e = nbn * (token tiles of experts < e)
    // (offsets null: one matrix, E = 1, of all A rows -- a dense projection)
    const int my_off = lane < p.E && p.offsets ? p.offsets[lane] : 0;
    const int my_rows = lane < p.E ? (p.offsets ? p.offsets[lane + 1] - my_off : (int)p.A) : 0;
    // complete on every path, so that no later counter wait is placed for them
    wait_vmem<0>();
    const int my_tiles = (my_rows >= p.mlo && my_rows <= p.mhi) ? (my_rows + C::BM - 1) / C::BM : 0;
    int in_tiles = my_tiles;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int v = __shfl_up(in_tiles, o, 64);
        if (lane >= o) in_tiles += v;
    }
    const int xcd = blockIdx.x & 7;
    const int per_xcd = gridDim.x >> 3;
    const int local = blockIdx.x >> 3;
    const int nk = p.K / C::BK;
    // items: expert, reduction part, weight block, token tile
    // (values read from one lane are uniform; readfirstlane keeps them, and
    // the step counts and branches derived from them, in scalar registers)
    auto uni = [](int v) { return __builtin_amdgcn_readfirstlane(v); };
    const int all_tiles = uni(__shfl(in_tiles, p.E - 1, 64));
    const int nparts = (UP || p.tail) ? 1 : uni(down_parts(nbn * all_tiles, per_xcd, nk, p.A, p.N, p.ksplit_max));
    if (!UP && p.ksplit_out && blockIdx.x == 0 && tid == 0) *p.ksplit_out = nparts;
    const int ex_items = nparts * nbn * (in_tiles - my_tiles);
    const int total = nparts * nbn * all_tiles;
    // The items are cut into 8 contiguous ranges of about equal cost, one per
    // XCD (equal counts leave the XCD whose experts end in full tiles with
    // the most work: an expert's last token tile of a few rows costs a
    // fraction of a full one).  Cost per (part, weight block) of expert e:
    // its full tiles plus its last tile by the blocks it multiplies.
    const int last_rows = my_tiles > 0 ? my_rows - C::BM * (my_tiles - 1) : 0;
    const int cnb = my_tiles > 0 ? kFullTileCost * (my_tiles - 1) + tile_cost(last_rows) : 0;
    const int64_t ce = (int64_t)nparts * nbn * cnb;
    int64_t cin = ce;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t v = __shfl_up(cin, o, 64);
        if (lane >= o) cin += v;
    }
    const int64_t cbefore = cin - ce;
    const int64_t ctot = __shfl(cin, p.E - 1, 64);
    // the first item whose cost prefix (at its start) is >= B
    auto first_item_at = [&](int64_t B) -> int {
        const uint64_t le = __ballot(lane < p.E && my_tiles > 0 && cbefore <= B);
        if (!le) return 0;
        const int ee = 63 - __builtin_clzll(le);
        const int64_t rel = B - __shfl(cbefore, ee, 64);
        const int cnb_e = __shfl(cnb, ee, 64);
        const int mt_e = __shfl(my_tiles, ee, 64);
        const int groups = nparts * nbn;
        const int ex = __shfl(ex_items, ee, 64);
        if (rel >= (int64_t)groups * cnb_e) return ex + groups * mt_e;
        int blk = (int)(rel / cnb_e);
        const int r2 = (int)(rel - (int64_t)blk * cnb_e);
        int m = (r2 + kFullTileCost - 1) / kFullTileCost;  // tile m starts at m * kFullTileCost
        if (m > mt_e - 1) {
            ++blk;
            m = 0;
        }
        return ex + blk * mt_e + m;
    };
    // The workgroups of an XCD take its items in rounds (workgroup j: items
    // j, j + P, j + 2P, ...).  DOWN with tail split: the items of whole
    // rounds of the grid are dealt in equal counts, XCD x taking the x-th
    // range; the rem < grid tiles left over would leave grid - rem
    // workgroups idle for a whole tile, so each of them is cut into `pieces`
    // = grid / rem reduction ranges spread over all the workgroups (piece g
    // to the g-th workgroup in XCD-major order, so the pieces of neighbouring
    // tiles of one weight block share an XCD); piece 0 writes the tile's
    // output as usual, the others write f32 pieces that fold_tail_kernel
    // adds to it.  Otherwise the ranges are of about equal cost and the last
    // round is left partial.
    const bool gtail = !UP && p.tail;
    const int grounds = gtail ? total / (int)gridDim.x : 0;
    // With the tail split the items are ordered in two classes: first every
    // tile but the experts' short last tiles (cost below a full tile), then
    // those short tiles.  The whole rounds then hold full-cost tiles where
    // they can, and the short ones (a few rows streaming a whole weight
    // block) go to the split tail; each class is expert-major, a weight
    // block's token tiles next to each other.
    const int short_e = (gtail && my_tiles > 0 && tile_cost(last_rows) < kFullTileCost) ? 1 : 0;
    const int a_tiles = my_tiles - short_e;
    int in_a = nbn * a_tiles, in_b = nbn * short_e;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int va = __shfl_up(in_a, o, 64);
        const int vb = __shfl_up(in_b, o, 64);
        if (lane >= o) {
            in_a += va;
            in_b += vb;
        }
    }
    const int ex_a = in_a - nbn * a_tiles, ex_b = in_b - nbn * short_e;
    const int n_a = uni(__shfl(in_a, p.E - 1, 64));
    // (uniform by construction; readfirstlane lets the compiler see it, so the
    // item indices and everything derived from them stay in scalar registers)
    const int beg = gtail ? xcd * grounds * per_xcd
                          : __builtin_amdgcn_readfirstlane(first_item_at((ctot * xcd + 7) / 8));
    const int end = gtail ? beg + grounds * per_xcd
                          : __builtin_amdgcn_readfirstlane(
                                xcd == 7 ? total : first_item_at((ctot * (xcd + 1) + 7) / 8));
    const int n_xcd = end - beg;
    const int rounds = n_xcd / per_xcd;
    const int rem = gtail ? total - grounds * (int)gridDim.x : 0;
    // (at most one piece per reduction step: every piece has a step)
    const int pieces = rem > 0 ? min((int)gridDim.x / rem, nk) : 1;
    const int gpiece = xcd * per_xcd + local;  // this workgroup's tail piece
    const int units = gtail ? rounds + (gpiece < rem * pieces ? 1 : 0)
                            : (local < n_xcd ? (n_xcd - local + per_xcd - 1) / per_xcd : 0);
    int* const tail_tab = gtail
        ? reinterpret_cast<int*>(p.y_out + p.slice + (int64_t)gridDim.x * kTailPiece) : nullptr;
    if (tail_tab && blockIdx.x == 0 && tid == 0) tail_tab[4 * gridDim.x] = pieces > 1 ? rem : 0;

    // a token load covers 8 rows starting at a multiple of 8: lane l takes row
    // l / 8 and the global chunk stored at slot l % 8 (odd loads start at 8
    // mod 16); bf16 weight loads the same.  An 8-bit weight load covers 16
    // rows of 64 bytes: lane l takes row l / 4 and the global chunk stored at
    // slot l % 4 (chunk c of row r lives at slot c ^ ((r >> 2) & 3)).
    const int lrow = lane >> 3;
    const int lchunk[2] = {(lane & 7) ^ ((lrow >> 1) & 7), (lane & 7) ^ (((8 + lrow) >> 1) & 7)};
    const int lchunk8 = (lane & 3) ^ ((lane >> 4) & 3);
    // Fragment reads: row (tile base + lane % 32); the tile bases are
    // multiples of 32, so the swizzles depend on the lane only.  bf16: k-step
    // ks of both operands is chunk 2 ks + lane / 32 of the row.  8-bit weights
    // order a step's reduction differently, identically for both operands:
    // k-step ks, lane half h = lane / 32 holds elements 32 h + 8 ks .. + 7,
    // so one 16-byte read of a weight row (chunk 2 h + p) serves k-steps 2p
    // and 2p + 1, and the token row's k-step ks is its chunk 4 h + ks.
    int xk[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        const int ch = F8 ? 4 * (lane >> 5) + ks : 2 * ks + (lane >> 5);
        xk[ks] = (lane & 31) * C::ROWB + ((ch ^ (((lane & 31) >> 1) & 7)) << 4);
    }
    int xa[2];
#pragma unroll
    for (int q = 0; q < 2; ++q)
        xa[q] = (lane & 31) * C::AROWB + (((2 * (lane >> 5) + q) ^ (((lane & 31) >> 2) & 3)) << 4);
    // byte offset of this wave's nt-th 32-row weight tile in an A slot (UP:
    // nt < 2 are w1 rows, nt + 2 the same rows of w3), and of its token tiles
    const int a_wave = (UP ? wr * 64 : wr * 128) * C::AROWB;
    auto atile = [](int nt) { return (UP ? (nt >> 1) * (C::BN / 2) + (nt & 1) * 32 : nt * 32) * C::AROWB; };

    // ---- items ----------------------------------------------------------------
    //
    // Items follow each other without a break in the load stream: the last two
    // steps of an item load the first two steps of the workgroup's next item
    // into the ring slots the steady state would use.  The next item's first
    // step is complete everywhere after the barrier of its predecessor's last
    // step and its second one lands during the predecessor's epilogue, so no
    // barrier or prologue is needed between items.  What the next item's
    // loads depend on through memory (its gathered token rows; DOWN: the
    // output rows of its epilogue) is loaded when the item before it starts,
    // and its gate weights when it starts itself, before the first step's
    // counter wait, which completes them.  (Re-issuing these loads into the
    // registers of the previous item's makes the compiler wait for all loads
    // and stores in flight at that point, the previous epilogue's included.)
    // An item of fewer than 3 steps (tiny reductions) is followed by a drain,
    // a barrier and a fresh prologue.
    struct Item {
        int e, part, nb, k0, kn, row0, m0, Mp;
        int slot;      // DOWN tail split: this workgroup's piece slot, or -1 (output to y)
        int src[L];    // this lane's token rows of its L token loads (UP: gathered slot ids)
        int orow[4];   // DOWN: output row of each epilogue column block
        float gw[4];   // DOWN: its gate weight
    };
    // the uniform part of this workgroup's u-th unit of work: item
    // beg + local + u P, or in the tail-split round a piece of a tile
    auto index_item = [&](int u, Item& it) {
        int w = beg + local + u * per_xcd;
        int pc = 0, ti = 0;
        if (u == rounds && rem > 0) {
            ti = gpiece / pieces;
            pc = gpiece - ti * pieces;
            w = grounds * (int)gridDim.x + ti;
        }
        int e, part, nb, mtile;
        if (gtail) {
            // (one reduction part in the tail split)
            part = 0;
            if (w < n_a) {
                const uint64_t le = __ballot(lane < p.E && a_tiles > 0 && ex_a <= w);
                e = 63 - __builtin_clzll(le);
                const int ma = uni(__shfl(a_tiles, e, 64));
                const int r = w - uni(__shfl(ex_a, e, 64));
                nb = r / ma;
                mtile = r - nb * ma;
            } else {
                const int wb = w - n_a;
                const uint64_t le = __ballot(lane < p.E && short_e > 0 && ex_b <= wb);
                e = 63 - __builtin_clzll(le);
                nb = wb - uni(__shfl(ex_b, e, 64));
                mtile = uni(__shfl(my_tiles, e, 64)) - 1;
            }
        } else {
            const uint64_t le = __ballot(lane < p.E && my_tiles > 0 && ex_items <= w);
            e = 63 - __builtin_clzll(le);
            const int mt_e = uni(__shfl(my_tiles, e, 64));
            int r = w - uni(__shfl(ex_items, e, 64));
            part = r / (nbn * mt_e);
            r -= part * nbn * mt_e;
            nb = r / mt_e;
            mtile = r - nb * mt_e;
        }
        it.e = e;
        it.part = part;
        it.nb = nb;
        const bool tail_unit = u == rounds && rem > 0;
        const int np = tail_unit ? pieces : nparts;  // (tail split: nparts = 1)
        const int pp = tail_unit ? pc : part;
        it.k0 = (int)((int64_t)nk * pp / np);
        it.kn = (int)((int64_t)nk * (pp + 1) / np) - it.k0;
        it.slot = pc > 0 ? gpiece : -1;
        if (tail_unit && pc == 0 && pieces > 1 && tid == 0) {
            int* t = tail_tab + 4 * ti;
            t[0] = e;
            t[1] = nb;
            t[2] = mtile;
            t[3] = pieces;
        }
        it.row0 = uni(__shfl(my_off, e, 64));
        it.m0 = mtile * C::BM;
        it.Mp = min(C::BM, uni(__shfl(my_rows, e, 64)) - it.m0);
    };
    // the loads item `it` depends on: wave w loads token rows [64w, 64w + 64)
    // (rows past the expert's end repeat its last row); DOWN: the scatter row
    // of each column block of the epilogue (with NMT = ceil(rows / 64) blocks
    // per token wave, as the tile body below chooses)
    auto fetch_rows = [&](Item& it) {
#pragma unroll
        for (int i = 0; i < L; ++i) {
            const int tr = 64 * wave + 8 * i + lrow;
            const int rowm = it.row0 + it.m0 + (tr < it.Mp ? tr : it.Mp - 1);
            it.src[i] = (UP && p.gather) ? p.gather[rowm] : rowm;
        }
        if constexpr (!UP) {
            const int nmt = (it.Mp + 63) >> 6;
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const int mloc = (wm * nmt + mt) * 32 + (lane & 31);
                const int rrow = it.row0 + it.m0 + (mloc < it.Mp ? mloc : it.Mp - 1);
                it.orow[mt] = (p.topk_w && p.perm) ? p.perm[rrow] : rrow;
            }
        }
    };
    auto fetch_gates = [&](Item& it) {
        if constexpr (!UP) {
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) it.gw[mt] = (p.topk_w && p.perm) ? p.topk_w[it.orow[mt]] : 1.0f;
        }
    };
    // Load addresses: a uniform base per item (scalar registers) plus a
    // 32-bit per-lane byte offset.  Wave w loads weight rows [64w, 64w + 64)
    // of the item's block (64 consecutive rows of w1, w3 or w2); the lane's
    // offset inside them does not depend on the item.  Token rows: the
    // lane's row of each of its L loads times the row pitch (token buffers
    // stay below 4 GiB; the launchers check).
    uint32_t aoff[2];
#pragma unroll
    for (int q = 0; q < 2; ++q)
        aoff[q] = F8 ? (uint32_t)((lane >> 2) * p.K + lchunk8 * 16) : (uint32_t)(lrow * p.K * 2 + lchunk[q] * 16);
    auto abase_of = [&](const Item& it) -> const unsigned char* {
        const bool a_second = UP && 64 * wave >= C::BN / 2;
        const int64_t wrow = (int64_t)it.e * p.N + it.nb * C::NOUT + 64 * wave - (a_second ? C::BN / 2 : 0);
        const unsigned char* wm8 = F8 ? (a_second ? p.qb : p.qa)
                                      : reinterpret_cast<const unsigned char*>(a_second ? p.wb : p.wa);
        return wm8 + (wrow * p.K + (int64_t)it.k0 * C::BK) * (F8 ? 1 : 2);
    };
    auto boff_of = [&](const Item& it, int i) -> uint32_t {
        const uint32_t src = (UP && p.gather) ? (uint32_t)it.src[i] / (uint32_t)p.kslots : (uint32_t)it.src[i];
        return src * (uint32_t)(p.K * 2) + (uint32_t)(lchunk[i & 1] * 16);
    };
    const unsigned char* const bbase = reinterpret_cast<const unsigned char*>(p.act);

    // The loads in flight come from one item at a time: la / lbk0 / lb
    // address its step 0, and step s of the running item is its step
    // s - lsh, clamped to its last step lkn - 1 (steps past the end re-load
    // the last one, so that the number of loads in flight, and with it every
    // counter wait, is the same in every step).
    const unsigned char* la = nullptr;
    int lbk0 = 0;
    uint32_t lb[L];
    int lsh = 0, lkn = 1;
    uint32_t nbo[L];  // the next item's token row offsets
    // bytes between a wave's consecutive weight loads (8 or 16 rows)
    const int64_t astep = (int64_t)16 * p.K;
    auto load_a = [&](int slot, int s, int i) {
        const int st = min(s - lsh, lkn - 1);
        const unsigned char* base = la + (int64_t)st * C::BK * (F8 ? 1 : 2) + i * astep;
        const int rows = F8 ? 16 : 8;
        __builtin_amdgcn_global_load_lds(
            (const void __attribute__((address_space(1)))*)(base + aoff[F8 ? 0 : (i & 1)]),
            (void __attribute__((address_space(3)))*)(ring + slot + (64 * wave + rows * i) * C::AROWB),
            16, 0, 0);
    };
    auto load_b = [&](int slot, int s, int i) {
        const int st = min(s - lsh, lkn - 1);
        const unsigned char* base = bbase + (int64_t)(lbk0 + st) * C::BK * 2;
        __builtin_amdgcn_global_load_lds(
            (const void __attribute__((address_space(1)))*)(base + lb[i]),
            (void __attribute__((address_space(3)))*)(ring + C::B_OFF + slot + (64 * wave + 8 * i) * C::ROWB),
            16, 0, 0);
    };
    // ring slots (byte offsets) of A(j), A(j+1), A(j+2) and of B(j), B(j+1)
    // during step j; they rotate at the end of every step and carry over from
    // one item to the next
    int sa0 = 0, sa1 = C::ASLOT, sa2 = 2 * C::ASLOT;
    int sb0 = 0, sb1 = C::SLOT;
    // steps 0 and 1 of `it` into the slots of A(0), A(1), B(0), B(1), by every
    // wave, then complete everywhere
    // (from_next: the token offsets were computed into nbo during the item
    // before)
    auto prologue = [&](const Item& it, bool from_next) {
        la = abase_of(it);
        lbk0 = it.k0;
#pragma unroll
        for (int i = 0; i < L; ++i) lb[i] = from_next ? nbo[i] : boff_of(it, i);
        lsh = 0;
        lkn = it.kn;
#pragma unroll
        for (int i = 0; i < LA; ++i) load_a(sa0, 0, i);
#pragma unroll
        for (int i = 0; i < LA; ++i) load_a(sa1, 1, i);
#pragma unroll
        for (int i = 0; i < L; ++i) load_b(sb0, 0, i);
#pragma unroll
        for (int i = 0; i < L; ++i) load_b(sb1, 1, i);
        wait_vmem<0>();
        __syncthreads();
    };

    Item cur, nxt;
    int u = 0;
    bool more = false, pipe = false;

    // The tile body for NMT multiplied 32-token column blocks per wave
    // (4: full tile).  The tile's blocks that hold rows are split evenly
    // between the two token waves: wave wm multiplies blocks
    // [wm NMT, wm NMT + NMT), NMT = ceil(blocks / 2), so a tile of an
    // expert's last few rows (or of an expert with 65-192 rows) skips the
    // MFMAs and fragment reads of empty blocks and both waves finish
    // together.  Only computed blocks are stored; columns past the rows
    // hold copies of the last row (see epilogue).
    auto tile = [&](auto nmt_tag) {
        constexpr int NMT = decltype(nmt_tag)::value;
        const int kn = cur.kn;
        const int b_wave = wm * NMT * 32 * C::ROWB;
        // token rows [0, 64 NMT) are multiplied: wave w loads rows
        // [64w, 64w + 64), so waves w >= NMT skip this item's token loads
        // (in a full tile every wave loads, with no branch) -- but not the
        // next item's.  The counter waits stay exact for them: the loads
        // younger than the ones a wait is for are A loads, which every wave
        // issues.
        bool bl = NMT == 4 || wave < NMT;
        lsh = 0;
        lkn = kn;
        floatx16 acc[NT][NMT];
#pragma unroll
        for (int i = 0; i < NT; ++i)
#pragma unroll
            for (int j = 0; j < NMT; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

        bf16x8 fa[2][NT], fb[2][NMT];
        // 8-bit weights: raw 16-byte reads, k-steps (0,1) and (2,3).  A
        // native vector type: an aggregate (HIP's uint4) load carries no
        // memory operand the compiler can tell apart from the in-flight
        // global->LDS loads, and it then waits for all of them (vmcnt(0))
        // before each read.
        u32x4 fq[NT][2];
        // fragment f (0 .. NT-1: weight tiles, NT ..: token tiles) of
        // k-step ks from the A slot as / B slot bs
        auto fread1 = [&](int as, int bs, int ks, int slot, int f) {
            if (f < NT) {
                fa[slot][f] = *reinterpret_cast<const bf16x8*>(ring + as + a_wave + xk[ks] + atile(f));
            } else {
                fb[slot][f - NT] = *reinterpret_cast<const bf16x8*>(
                    ring + C::B_OFF + bs + b_wave + xk[ks] + (f - NT) * 32 * C::ROWB);
            }
        };
        // 8-bit weights: token fragment m of k-step ks, and the raw weight
        // bytes of k-step pair q for tile nt
        auto fread_b = [&](int bs, int ks, int slot, int m) {
            fb[slot][m] = *reinterpret_cast<const bf16x8*>(ring + C::B_OFF + bs + b_wave + xk[ks] +
                                                           m * 32 * C::ROWB);
        };
        auto fread_q = [&](int as, int q, int nt) {
            fq[nt][q] = *reinterpret_cast<const u32x4*>(ring + as + a_wave + xa[q] + atile(nt));
        };
        auto fence = [] { __builtin_amdgcn_sched_barrier(0); };

        // Loads whose values the epilogue needs, issued before the first
        // step's loads so that its counter wait completes them: 8-bit
        // weights' row scales of this lane's accumulator rows (UP: w1 then
        // w3 rows of its two 32-row tiles; DOWN: its four tiles), and DOWN's
        // gate weights (their rows were loaded with the item before).
        floatx4 sc[4][4];
        if constexpr (F8) {
            const int n0 = cur.nb * C::NOUT + (UP ? wr * 64 : wr * 128) + 4 * (lane >> 5);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const float* sp = UP ? (t < 2 ? p.sa : p.sb) + (int64_t)cur.e * p.N + n0 + (t & 1) * 32
                                     : p.sa + (int64_t)cur.e * p.N + n0 + t * 32;
#pragma unroll
                for (int q = 0; q < 4; ++q) sc[t][q] = *reinterpret_cast<const floatx4*>(sp + 8 * q);
            }
        }
        fetch_gates(cur);

        // k-step 0 of step 0: A(0) and B(0) are complete everywhere (the
        // prologue's barrier, or the previous item's last step)
        if constexpr (F8) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) fread_q(sa0, 0, nt);
#pragma unroll
            for (int m = 0; m < NMT; ++m) fread_b(sb0, 0, 0, m);
        } else {
#pragma unroll
            for (int f = 0; f < NT + NMT; ++f) fread1(sa0, sb0, 0, 0, f);
        }

        // Step j, k-step ks: its NT x NMT MFMAs use the fragments in
        // register slot ks & 1, and memory operations follow the MFMAs:
        // first the reads of the next k-step's fragments into the other
        // slot, two per MFMA (so they are complete long before that k-step
        // starts), then this k-step's share of the loads: A(j+2) in k-steps 0 and 1, B(j+2) in
        // k-step 3.  8-bit weights read their raw bytes a pair of k-steps
        // at a time (k-step 0: pair 1 of step j; k-step 3: pair 0 of step
        // j+1) and widen them to bf16 before the MFMAs of each weight tile.
        // After k-step 2 every wave waits for its reads of step j's last
        // fragments and for its loads up to B(j+1) (loads retire in order;
        // only A(j+2) may stay in flight), then one barrier makes A(j+1)
        // and B(j+1) complete for all waves and frees the slots of A(j)
        // and B(j): B(j+2) takes B(j)'s slot in k-step 3 and A(j+3) A(j)'s
        // in the next step.  From step kn - 2 on, "step j + 2" is step
        // j + 2 - kn of the next item.  (A do-while: the body runs at least
        // once, so the compiler's counter tracking sees every value loaded
        // before it as complete after the first step's wait.)
        int j = 0;
        do {
            if (pipe && j == kn - 2) {
                la = abase_of(nxt);
                lbk0 = nxt.k0;
#pragma unroll
                for (int i = 0; i < L; ++i) lb[i] = nbo[i];
                lsh = kn;
                lkn = nxt.kn;
                bl = true;
            }
            static_for<4>([&](auto ks_tag) {
                constexpr int ks = decltype(ks_tag)::value;
                constexpr int cur_s = ks & 1;
                constexpr int rk = ks < 3 ? ks + 1 : 0;  // the k-step read next
                const int ras = ks < 3 ? sa0 : sa1;       // ... from these slots
                const int rbs = ks < 3 ? sb0 : sb1;
                constexpr int M = NT * NMT;
                constexpr int NR = F8 ? NMT + ((ks == 0 || ks == 3) ? NT : 0) : NT + NMT;
                constexpr int NLD = (ks == 0 || ks == 1) ? LA / 2 : (ks == 3 ? L : 0);
                constexpr int X = NR + NLD;
                auto extra = [&](auto x_tag) {
                    constexpr int x = decltype(x_tag)::value;
                    if constexpr (x < NR) {
                        if constexpr (F8) {
                            if constexpr (x < NMT)
                                fread_b(rbs, rk, cur_s ^ 1, x);
                            else if constexpr (ks == 0)
                                fread_q(sa0, 1, x - NMT);
                            else
                                fread_q(sa1, 0, x - NMT);
                        } else {
                            fread1(ras, rbs, rk, cur_s ^ 1, x);
                        }
                    } else if constexpr (ks == 3) {
                        if (bl) load_b(sb0, j + 2, x - NR);
                    } else {
                        load_a(sa2, j + 2, ks * (LA / 2) + (x - NR));
                    }
                };
                bf16x8 a;
                static_for<M>([&](auto i_tag) {
                    constexpr int i = decltype(i_tag)::value;
                    constexpr int g = i / NMT, m = i % NMT;
                    if constexpr (m == 0) {
                        if constexpr (F8) {
                            const u32x4 q = fq[g][ks >> 1];
                            a = (ks & 1) ? e4m3x8_to_bf16(q[2], q[3]) : e4m3x8_to_bf16(q[0], q[1]);
                        } else {
                            a = fa[cur_s][g];
                        }
                    }
                    acc[g][m] = mfma32x32x16(a, fb[cur_s][m], acc[g][m]);
                    // the fragment reads two after each of the first MFMAs,
                    // then the loads spread over the remaining ones: the
                    // next k-step waits for all of this one's reads, and
                    // reads issued one per MFMA left too little time for
                    // them behind the other waves' reads and the
                    // global->LDS writes (prefill up GEMM 3.7% slower)
                    static_for<X>([&](auto x_tag) {
                        constexpr int x = decltype(x_tag)::value;
                        constexpr int h = (NR + 1) / 2;
                        constexpr int at = x < NR ? x / 2 : h + (x - NR) * (M - h) / (NLD > 0 ? NLD : 1);
                        static_assert(at < M, "every extra follows an MFMA");
                        if constexpr (at == i) extra(x_tag);
                    });
                    fence();
                });
                if constexpr (ks == 2) {
                    wait_lds();
                    wait_vmem<LA>();
                    fence();
                    __builtin_amdgcn_s_barrier();
                    fence();
                    // the next item's token rows were loaded before this
                    // item's first step and are complete now
                    if (more && j == 0) {
#pragma unroll
                        for (int i = 0; i < L; ++i) nbo[i] = boff_of(nxt, i);
                    }
                }
            });
            const int ta = sa0;
            sa0 = sa1;
            sa1 = sa2;
            sa2 = ta;
            const int tb = sb0;
            sb0 = sb1;
            sb1 = tb;
        } while (++j < kn);

        // epilogue: lane holds, per 32x32 tile, column (token) lane % 32 and
        // rows (weight rows) 8q + 4 * (lane / 32) + i, q, i < 4.  Straight-line
        // code, one output tile at a time: any branch here makes the compiler
        // copy all accumulators out of their registers at once.  Token columns
        // past the expert's rows were loaded from its last row, so they hold
        // exactly that row's results and store the same bits to the same place.
        // 8-bit weights: each weight row's scale multiplies its accumulators.
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) {
            if (UP) {
                const int mloc = (wm * NMT + mt) * 32 + (lane & 31);
                const int64_t rrow = cur.row0 + cur.m0 + (mloc < cur.Mp ? mloc : cur.Mp - 1);
                const int n0 = cur.nb * C::NOUT + wr * 64 + 4 * (lane >> 5);
                bf16_t* hrow = p.h_out + rrow * p.N + n0;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    // the accumulators are redefined here (in their AGPRs), so
                    // their copies into VGPRs cannot move above this point
                    asm volatile("" : "+a"(acc[h][mt]), "+a"(acc[h + 2][mt]));
                    floatx16 u = acc[h][mt];
                    floatx16 v = acc[h + 2][mt];
                    if constexpr (F8) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                u[4 * q + i] *= sc[h][q][i];
                                v[4 * q + i] *= sc[h + 2][q][i];
                            }
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        uint2 pk;
                        pk.x = pack_bf16x2(silu(u[4 * q + 0]) * v[4 * q + 0], silu(u[4 * q + 1]) * v[4 * q + 1]);
                        pk.y = pack_bf16x2(silu(u[4 * q + 2]) * v[4 * q + 2], silu(u[4 * q + 3]) * v[4 * q + 3]);
                        *reinterpret_cast<uint2*>(hrow + h * 32 + 8 * q) = pk;
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else {
                int orow_mt = cur.orow[mt];
                float gw = cur.gw[mt];
                // (kept here: computed before the steps, the row addresses
                // would occupy registers through all of them)
                asm volatile("" : "+v"(orow_mt), "+v"(gw));
                const int64_t orow = orow_mt;
                const int n0 = cur.nb * C::NOUT + wr * 128 + 4 * (lane >> 5);
                // (a split tile's later pieces: tile-local rows of 256 in
                // this workgroup's slot; a select, not a branch)
                const int mloc = (wm * NMT + mt) * 32 + (lane & 31);
                float* const ypiece = p.y_out + p.slice + (int64_t)(cur.slot < 0 ? 0 : cur.slot) * kTailPiece +
                                      mloc * 256 + (n0 - cur.nb * C::NOUT);
                float* const yout = p.y_out + cur.part * p.slice + orow * p.N + n0;
                float* yrow = cur.slot < 0 ? yout : ypiece;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    asm volatile("" : "+a"(acc[nt][mt]));
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        floatx4 g4 = {gw, gw, gw, gw};
                        if constexpr (F8) g4 = g4 * sc[nt][q];
                        float4 v;
                        v.x = g4[0] * acc[nt][mt][4 * q + 0];
                        v.y = g4[1] * acc[nt][mt][4 * q + 1];
                        v.z = g4[2] * acc[nt][mt][4 * q + 2];
                        v.w = g4[3] * acc[nt][mt][4 * q + 3];
                        *reinterpret_cast<float4*>(yrow + nt * 32 + 8 * q) = v;
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };
    static_assert(MT == 4, "the tile variants cover 1 to 4 blocks per wave");

    if (units == 0) return;
    index_item(0, cur);
    fetch_rows(cur);
    prologue(cur, false);
    while (true) {
        more = u + 1 < units;
        if (more) {
            index_item(u + 1, nxt);
            fetch_rows(nxt);
        }
        pipe = more && cur.kn >= 3;
        if (cur.Mp <= 64)
            tile(std::integral_constant<int, 1>{});
        else if (cur.Mp <= 128)
            tile(std::integral_constant<int, 2>{});
        else if (cur.Mp <= 192)
            tile(std::integral_constant<int, 3>{});
        else
            tile(std::integral_constant<int, 4>{});
        if (!more) break;
        if (!pipe) {
            // the ring is reused from scratch: this item's tail loads and
            // stores done, every wave past its last read
            wait_vmem<0>();
            __syncthreads();
            prologue(nxt, true);
        }
        cur = nxt;
        ++u;
    }
    // no global->LDS load may still be in flight when the workgroup ends
    wait_vmem<0>();
}

// Adds the later pieces of every tile that the down GEMM split in its last
// round (table written by the tiles' first pieces) to the tile's output in
// y: rows scattered through perm as in the down epilogue, the gate weights
// already applied, pieces added in order after piece 0's value.  Workgroup
// (split tile i, block of 16 rows) (grid = the down launch's grid x 16);
// each thread 4 rows of one 16-byte column chunk, all loads of a row issued
// together.
constexpr int kFoldRows = 16;
__global__ __launch_bounds__(256) void fold_tail_kernel(float* __restrict__ y, int64_t slice,
                                                        const int32_t* __restrict__ offsets,
                                                        const int32_t* __restrict__ perm,
                                                        const float* __restrict__ topk_w, int N,
                                                        int q_grid)
{
    const int i = blockIdx.x / (256 / kFoldRows);
    const int rb = blockIdx.x - i * (256 / kFoldRows);
    const float* pieces = y + slice;
    const int* tab = reinterpret_cast<const int*>(pieces + (int64_t)q_grid * kTailPiece);
    if (i >= tab[4 * q_grid]) return;
    const int e = tab[4 * i], nb = tab[4 * i + 1], mtile = tab[4 * i + 2], np = tab[4 * i + 3];
    const int row0 = offsets[e] + mtile * 256;
    const int Mp = min(256, offsets[e + 1] - row0);
    const int c4 = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < kFoldRows / 4; ++j) {
        const int lr = rb * kFoldRows + 4 * j + (threadIdx.x >> 6);
        if (lr >= Mp) continue;
        const int64_t a = (topk_w && perm) ? perm[row0 + lr] : row0 + lr;
        float4* yr = reinterpret_cast<float4*>(y + a * N + nb * 256) + c4;
        float4 v = *yr;
        for (int pc = 1; pc < np; ++pc) {
            // piece pc of split tile i has slot i np + pc
            const int slot = i * np + pc;
            const float4 w =
                reinterpret_cast<const float4*>(pieces + (int64_t)slot * kTailPiece + lr * 256)[c4];
            v.x += w.x;
            v.y += w.y;
            v.z += w.z;
            v.w += w.w;
        }
        *yr = v;
    }
}

// persistent grid: one workgroup per CU, fewer for fewer items (a bound:
// the real tile counts are on the device), a multiple of the 8 XCDs
template <bool UP>
int q_grid(int N, int E, int64_t A, int ksplit_max)
{
    using C = QCfg<UP, false>;  // the item shape does not depend on the weight format
    const int64_t nbn = N / C::NOUT;
    const int64_t items = nbn * (A / C::BM + E) * (UP ? 1 : ksplit_max);
    int64_t grid = cu_count();
    if (grid > items) grid = items;
    return static_cast<int>(((grid + 7) / 8) * 8);
}

template <bool UP, bool F8>
hipError_t run_q(const TiledParams& p, int64_t A, hipStream_t stream)
{
    using C = QCfg<UP, F8>;
    // the dynamic-LDS limit is set once per device and kernel instance; the
    // flags are per device and set under a lock, so concurrent first calls
    // from several threads or on several devices are safe
    static std::atomic<bool> attr_set[kMaxDevices];
    static std::mutex attr_mu;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices || !attr_set[dev].load(std::memory_order_acquire)) {
        std::lock_guard<std::mutex> lk(attr_mu);
        if (dev < 0 || dev >= kMaxDevices || !attr_set[dev].load(std::memory_order_relaxed)) {
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(&q_kernel<UP, F8>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
            if (e != hipSuccess) return e;
            if (dev >= 0 && dev < kMaxDevices) attr_set[dev].store(true, std::memory_order_release);
        }
    }
    const int grid = q_grid<UP>(p.N, p.E, A, p.ksplit_max);
    q_kernel<UP, F8><<<static_cast<unsigned>(grid), C::THREADS, C::LDS_BYTES, stream>>>(p);
    return hipGetLastError();
}

int cu_count()
{
    static std::atomic<int> cached[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (!n) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

}  // namespace

// rows: token rows of the largest activation buffer the tiled kernels read
// (x, the permuted rows or h); they address it with 32-bit byte offsets
bool tiled_supported(int d, int ffn, int64_t rows)
{
    return ffn % QCfg<true, false>::NOUT == 0 && d % QCfg<false, false>::NOUT == 0 &&
           d % QCfg<true, false>::BK == 0 && ffn % QCfg<false, false>::BK == 0 &&
           rows * 2 * (d > ffn ? d : ffn) < (int64_t(1) << 32);
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
    p.ksplit_max = 1;
    p.A = a.A;
    return a.q1 ? run_q<true, true>(p, a.A, stream) : run_q<true, false>(p, a.A, stream);
}

int tiled_down_grid(const DownArgs& a)
{
    return q_grid<false>(a.d, a.E, a.A, a.ksplit_max > 1 ? a.ksplit_max : 1);
}

hipError_t launch_tiled_down(const DownArgs& a, hipStream_t stream)
{
    TiledParams p{};
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
    p.mlo = a.mlo;
    p.mhi = a.mhi;
    p.ksplit_max = a.ksplit_max > 1 ? a.ksplit_max : 1;
    p.slice = a.A * a.d;
    p.ksplit_out = a.ksplit_out;
    p.A = a.A;
    // Tail split where the caller's slices 1.. hold a piece per workgroup and
    // the table (the prefill shapes): the tiles stay uncut, so the combine
    // reads one slice; otherwise the reduction may be cut into uniform parts.
    const int grid = q_grid<false>(a.d, a.E, a.A, p.ksplit_max);
    p.tail = (p.ksplit_max >= 4 && a.ksplit_out && a.offsets &&
              (int64_t)(p.ksplit_max - 1) * p.slice >= (int64_t)grid * kTailPiece + 4 * grid + 8)
                 ? 1 : 0;
    hipError_t e = a.q2 ? run_q<false, true>(p, a.A, stream) : run_q<false, false>(p, a.A, stream);
    if (e != hipSuccess || !p.tail) return e;
    fold_tail_kernel<<<static_cast<unsigned>(grid * (256 / kFoldRows)), 256, 0, stream>>>(
        a.y, p.slice, a.offsets, a.topk_w ? a.perm : nullptr, a.topk_w, a.d, grid);
    return hipGetLastError();
}

}  // namespace moe
