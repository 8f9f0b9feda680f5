// Router GEMM, top-k gating and token-to-expert dispatch for gfx950.
//
// The router of a Mixtral MoE layer (the model of the paper's engine, Sec. 4.1)
// scores every token against every expert, keeps the k best experts and
// weights them with a softmax over the kept scores.  Here:
//   * up to 256 tokens (and for more than 16 experts): one workgroup (8
//     wave64) per token, or per 64 / E tokens for long inputs: each lane
//     multiplies 16-byte chunks of x against the same chunk of every
//     expert's router row, accumulating in f32; the per-(token, expert)
//     partial sums are combined by a transposed wave butterfly and a
//     fixed-order sum over the waves, so results are bitwise reproducible and
//     the same for any tokens per workgroup;
//   * more tokens, up to 16 experts: 16 tokens per workgroup on the matrix
//     cores (16x16x32 bf16 MFMAs, f32 accumulation), the reduction split over
//     16 waves and their partial tiles summed in a fixed order;
//   * the top k are then ranked on the key (logit, -expert) -- equal logits
//     pick the lower expert -- by k arg-max butterflies over each token's
//     expert lanes (up to 16 experts; one lane per token in the matrix-core
//     kernel), or by a wave-wide arg-max butterfly for more, and the softmax
//     over the selected logits is formed in f32;
//   * a single-workgroup dispatch kernel builds the expert histogram, its
//     exclusive scan and the stable expert-major permutation: up to 1024
//     assignments one per thread (LDS-atomic histogram, ranks among equal
//     experts by wave ballots), more eight per thread (packed per-thread
//     counts and wave prefix sums).
#include "common.hpp"
#include "launch.hpp"

#include <math.h>

namespace moe {

namespace {

constexpr int ROUTE_THREADS = 512;  // one 16-byte chunk per lane at d = 4096

struct Cand {
    float v;
    int i;
};

__device__ __forceinline__ bool ahead(const Cand& a, const Cand& b)
{
    return a.v > b.v || (a.v == b.v && a.i < b.i);
}

// The ranking key of a logit: a NaN (non-finite input, outside the defined
// domain) ranks as -inf, so the order stays total, every selected id is a
// real expert of this token, and the token's gates come out NaN instead of
// its routing reaching other tokens' rows.
__device__ __forceinline__ float rank_key(float v) { return v != v ? -INFINITY : v; }

// TPB tokens per workgroup pass (EMAX * TPB <= 64): every 16-byte chunk of the
// router rows is loaded once and multiplied with the TPB tokens' chunks, and
// the (token, expert) partial sums are reduced together.  A sum's order does
// not depend on TPB or on the token's place in the pass (the same chunks per
// lane in the same order, the same lane tree, the same wave order), so the
// logits are bitwise those of one token per workgroup.
template <int EMAX, int TPB>
__global__ __launch_bounds__(ROUTE_THREADS) void router_topk_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, const float* __restrict__ bias,
    int64_t T, int d, int E, int k, int32_t* __restrict__ topk_ids, float* __restrict__ topk_w,
    float* __restrict__ logits_out)
{
    constexpr int NV = EMAX * TPB;  // (token, expert) sums per lane, index j * EMAX + e
    static_assert(NV <= 64 && (NV & (NV - 1)) == 0, "at most 64 sums, a power of two");
    __shared__ float red[ROUTE_THREADS / 64][NV];
    __shared__ float lg[TPB][EMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nchunk = d >> 3;  // 16-byte chunks per row
    const int64_t npass = (T + TPB - 1) / TPB;
    // the bias of the sum this thread finishes (loaded with the first
    // operands, not after the reduction)
    const float bias_e = (bias && tid < NV && tid % EMAX < E) ? bias[tid % EMAX] : 0.0f;

    for (int64_t pass = blockIdx.x; pass < npass; pass += gridDim.x) {
        const int64_t t0 = pass * TPB;
        const int nt = static_cast<int>(T - t0 < TPB ? T - t0 : TPB);
        float acc[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) acc[i] = 0.0f;
        for (int c = tid; c < nchunk; c += ROUTE_THREADS) {
            float wf[EMAX][8];
#pragma unroll
            for (int e = 0; e < EMAX; ++e) {
                if (e < E) {
                    const uint4 wv = ldg16(wr + (int64_t)e * d + c * 8);
                    const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        wf[e][2 * q] = __uint_as_float(ww[q] << 16);
                        wf[e][2 * q + 1] = __uint_as_float(ww[q] & 0xffff0000u);
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < TPB; ++j) {
                if (j < nt) {
                    const uint4 xv = ldg16(x + (t0 + j) * (int64_t)d + c * 8);
                    float xf[8];
                    const uint32_t xw[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        xf[2 * q] = __uint_as_float(xw[q] << 16);
                        xf[2 * q + 1] = __uint_as_float(xw[q] & 0xffff0000u);
                    }
#pragma unroll
                    for (int e = 0; e < EMAX; ++e) {
                        if (e < E) {
                            float s = acc[j * EMAX + e];
#pragma unroll
                            for (int q = 0; q < 8; ++q) s = fmaf(xf[q], wf[e][q], s);
                            acc[j * EMAX + e] = s;
                        }
                    }
                }
            }
        }
        // Transposed butterfly: at each exchange a lane keeps half of its
        // partial sums and ships the other half to its partner, so after
        // log2(NV) exchanges lane l holds sum l / (64/NV) over 2^log2(NV)
        // lanes; the remaining lane bits are then folded.  Every sum is
        // reduced over the same lane tree (bit 5 first, then 4, ... 0).
        float v[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) v[i] = acc[i];
#pragma unroll
        for (int half = NV / 2, m = 32; half >= 1; half >>= 1, m >>= 1) {
            const bool hi = (lane & m) != 0;
#pragma unroll
            for (int i = 0; i < half; ++i) {
                const float send = hi ? v[i] : v[i + half];
                const float keep = hi ? v[i + half] : v[i];
                v[i] = keep + wave_shfl_xor(send, m);
            }
        }
        constexpr int LANES_PER_V = 64 / NV;
        float tot = v[0];
#pragma unroll
        for (int m = LANES_PER_V / 2; m >= 1; m >>= 1) tot += wave_shfl_xor(tot, m);
        if ((lane % LANES_PER_V) == 0) red[wave][lane / LANES_PER_V] = tot;
        __syncthreads();
        if (EMAX <= 16) {
            // few experts: wave 0's lane j * EMAX + e finishes the logit of
            // (token j, expert e), and k arg-max butterflies over each token's
            // EMAX lanes pick its experts on the key (logit, -expert), so an
            // equal logit keeps the lower index; no LDS round trip
            if (wave == 0) {
                const int j = lane / EMAX, e = lane - j * EMAX;
                const bool live = lane < NV && j < nt && e < E;
                Cand me;
                me.v = -INFINITY;
                me.i = 0x7fffffff;
                if (live) {
                    float s = red[0][lane];
#pragma unroll
                    for (int w = 1; w < ROUTE_THREADS / 64; ++w) s += red[w][lane];
                    if (bias) s += bias_e;
                    if (logits_out) logits_out[(t0 + j) * E + e] = s;
                    me.v = rank_key(s);
                    me.i = e;
                }
                float selv[8];
                int seli[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    if (q < k) {
                        Cand b = me;
#pragma unroll
                        for (int m = EMAX / 2; m >= 1; m >>= 1) {
                            Cand o;
                            o.v = wave_shfl_xor(b.v, m);
                            o.i = wave_shfl_xor(b.i, m);
                            if (ahead(o, b)) b = o;
                        }
                        selv[q] = b.v;
                        seli[q] = b.i;
                        if (live && e == b.i) {
                            me.v = -INFINITY;
                            me.i = 0x7fffffff;
                        }
                    }
                }
                if (e == 0 && j < nt) {
                    const int64_t t = t0 + j;
                    float ex[8], den = 0.0f;
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        if (q < k) {
                            ex[q] = expf(selv[q] - selv[0]);
                            den += ex[q];
                        }
                    }
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        if (q < k) {
                            topk_ids[t * k + q] = seli[q];
                            topk_w[t * k + q] = ex[q] / den;
                        }
                    }
                }
            }
            __syncthreads();
            continue;
        }
        if (tid < NV) {
            const int j = tid / EMAX, e = tid - j * EMAX;
            if (j < nt && e < E) {
                float s = red[0][tid];
#pragma unroll
                for (int w = 1; w < ROUTE_THREADS / 64; ++w) s += red[w][tid];
                if (bias) s += bias_e;
                lg[j][e] = s;
                if (logits_out) logits_out[(t0 + j) * E + e] = s;
            }
        }
        __syncthreads();
        // more experts: wave j ranks token j with a wave-wide arg-max
        if (wave < nt) {
            const int64_t t = t0 + wave;
            Cand me;
            me.v = lane < E ? rank_key(lg[wave][lane]) : -INFINITY;
            me.i = lane < E ? lane : 0x7fffffff;
            float selv[8];
            int seli[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                if (j < k) {
                    Cand b = me;
#pragma unroll
                    for (int m = 32; m >= 1; m >>= 1) {
                        Cand o;
                        o.v = wave_shfl_xor(b.v, m);
                        o.i = wave_shfl_xor(b.i, m);
                        if (ahead(o, b)) b = o;
                    }
                    selv[j] = b.v;
                    seli[j] = b.i;
                    if (lane == b.i) {
                        me.v = -INFINITY;
                        me.i = 0x7fffffff;
                    }
                }
            }
            if (lane == 0) {
                float den = 0.0f;
                float ex[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (j < k) {
                        ex[j] = expf(selv[j] - selv[0]);
                        den += ex[j];
                    }
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (j < k) {
                        topk_ids[t * k + j] = seli[j];
                        topk_w[t * k + j] = ex[j] / den;
                    }
                }
            }
        }
        __syncthreads();
    }
}

// Up to 16 experts: the router GEMM on the matrix cores.  A workgroup takes
// 16 tokens (one 16 x 16 output tile of 16x16x32 bf16 MFMAs: tokens x
// experts, experts past E multiplied by zeros); its 16 waves each take a
// contiguous sixteenth of the reduction and issue all of their operand loads
// before their MFMAs, so the tile costs one memory round trip, and the 16
// partial tiles are summed in wave order.  A token's logits therefore do not
// depend on the other tokens or on T.  Ranking and softmax as above, one
// lane per token.
constexpr int RM_WAVES = 16;
constexpr int RM_THREADS = RM_WAVES * 64;
constexpr int RM_UNROLL = 8;  // 32-element steps per wave loaded at once

__global__ __launch_bounds__(RM_THREADS) void router_mfma_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, const float* __restrict__ bias,
    int64_t T, int d, int E, int k, int32_t* __restrict__ topk_ids, float* __restrict__ topk_w,
    float* __restrict__ logits_out)
{
    __shared__ floatx4 part[RM_WAVES][64];
    __shared__ float lg[16][17];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int row = lane & 15, kq = lane >> 4;  // operand row (token / expert), 8-element quarter
    const int64_t t0 = (int64_t)blockIdx.x * 16;
    const int64_t t = t0 + row < T ? t0 + row : T - 1;  // rows past T repeat the last token
    const bool has_e = row < E;
    const bf16_t* xr = x + t * d + kq * 8;
    const bf16_t* wrow = wr + (int64_t)(has_e ? row : 0) * d + kq * 8;
    // wave 0 adds expert `row`'s bias after the reduction; loaded now
    const float bias_e = (wave == 0 && has_e && bias) ? bias[row] : 0.0f;
    const int nsteps = d >> 5;
    const int spw = (nsteps + RM_WAVES - 1) / RM_WAVES;
    const int s_beg = wave * spw;
    const int s_end = min(s_beg + spw, nsteps);
    floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int s0 = s_beg; s0 < s_end; s0 += RM_UNROLL) {
        bf16x8 a[RM_UNROLL], b[RM_UNROLL];
#pragma unroll
        for (int u = 0; u < RM_UNROLL; ++u) {
            const int s = s0 + u;
            if (s < s_end) {
                a[u] = as_bf16x8(ldg16(xr + s * 32));
                b[u] = has_e ? as_bf16x8(ldg16(wrow + s * 32)) : bf16x8{};
            }
        }
#pragma unroll
        for (int u = 0; u < RM_UNROLL; ++u)
            if (s0 + u < s_end) acc = mfma16x16x32(a[u], b[u], acc);
    }
    part[wave][lane] = acc;
    __syncthreads();
    // lane l of wave 0: tokens 4 (l / 16) + i, expert l % 16
    if (wave == 0) {
        floatx4 v = part[0][lane];
#pragma unroll
        for (int w = 1; w < RM_WAVES; ++w) v += part[w][lane];
        const int e = row;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int tr = 4 * kq + i;
            float l = v[i];
            if (e < E && bias) l += bias_e;
            lg[tr][e] = l;
            if (e < E && logits_out && t0 + tr < T) logits_out[(t0 + tr) * E + e] = l;
        }
    }
    __syncthreads();
    if (tid < 16 && t0 + tid < T) {
        const int64_t tt = t0 + tid;
        int seli[8];
        float selv[8];
        uint32_t taken = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < k) {
                int best = -1;
                float bv = 0.0f;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    if (e < E && !(taken & (1u << e))) {
                        const float le = rank_key(lg[tid][e]);
                        // strict: an equal logit keeps the lower index
                        if (best < 0 || le > bv) {
                            best = e;
                            bv = le;
                        }
                    }
                }
                taken |= 1u << best;
                seli[j] = best;
                selv[j] = bv;
            }
        }
        float ex[8], den = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < k) {
                ex[j] = expf(selv[j] - selv[0]);
                den += ex[j];
            }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < k) {
                topk_ids[tt * k + j] = seli[j];
                topk_w[tt * k + j] = ex[j] / den;
            }
        }
    }
}

constexpr int DISPATCH_THREADS = 1024;
constexpr int DISPATCH_WAVES = DISPATCH_THREADS / 64;

// One workgroup.  offsets[0..E], perm[0..A-1].
__global__ __launch_bounds__(DISPATCH_THREADS) void dispatch_kernel(
    const int32_t* __restrict__ ids, int64_t A, int E, int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm)
{
    __shared__ int cnt[64];
    __shared__ int base[64];    // running start of each expert's next rows
    __shared__ int wcnt[DISPATCH_WAVES][64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid < 64) cnt[tid] = 0;
    __syncthreads();
    // ids come from the router kernel and lie in [0, E); the clamp keeps a
    // corrupted id from indexing past the histogram
    auto expert_of = [&](int64_t a) { return min(max(ids[a], 0), E - 1); };
    for (int64_t a = tid; a < A; a += DISPATCH_THREADS) atomicAdd(&cnt[expert_of(a)], 1);
    __syncthreads();
    if (wave == 0) {
        int c = lane < E ? cnt[lane] : 0;
        int incl = c;
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) {
            int o = __shfl_up(incl, m, 64);
            if (lane >= m) incl += o;
        }
        if (lane < E) {
            base[lane] = incl - c;
            offsets[lane] = incl - c;
        }
        if (lane == E - 1) offsets[E] = incl;
    }
    __syncthreads();
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int64_t b0 = 0; b0 < A; b0 += DISPATCH_THREADS) {
        const int64_t a = b0 + tid;
        const int e = a < A ? expert_of(a) : -1;
        if (lane < 64) wcnt[wave][lane] = 0;
        // rank among lanes of this wave with the same expert
        int rank = 0;
        uint64_t todo = __ballot(e >= 0);
        while (todo) {
            const int leader = __ffsll(static_cast<unsigned long long>(todo)) - 1;
            const int le = __shfl(e, leader, 64);
            const uint64_t same = __ballot(e == le);
            if (e == le) rank = __popcll(same & lt_mask);
            if (lane == 0) wcnt[wave][le] = __popcll(same);
            todo &= ~same;
        }
        __syncthreads();
        if (e >= 0) {
            int before = 0;
            for (int w = 0; w < wave; ++w) before += wcnt[w][e];
            perm[base[e] + before + rank] = static_cast<int32_t>(a);
        }
        __syncthreads();
        if (tid < E) {
            int tot = 0;
            for (int w = 0; w < DISPATCH_WAVES; ++w) tot += wcnt[w][tid];
            base[tid] += tot;
        }
        __syncthreads();
    }
}

// Dispatch with 8 consecutive assignments per thread: one workgroup places
// up to 8192 assignments between two barriers.  Every thread counts its
// assignments per expert, packed three experts to a 32-bit word (10 bits
// each: a wave holds at most 512 of one expert), the waves take inclusive
// prefix sums of the packed words by shuffles, one wave scans the wave
// totals per expert, and each assignment goes to
//   offsets[e] + (chunks before) + (waves before) + (lanes before) + (its
//   rank among the thread's earlier assignments of e),
// which is the stable expert-major order.  Inputs longer than 8192
// assignments take a counting pass first and place chunk by chunk.
constexpr int D8_THREADS = 1024;
constexpr int D8_WAVES = D8_THREADS / 64;
constexpr int D8_PER = 8;
constexpr int D8_CHUNK = D8_THREADS * D8_PER;
constexpr int D8_MAXW = 22;  // packed words for up to 64 experts

template <int NW>
__device__ __forceinline__ void d8_pack(const int (&id)[D8_PER], uint32_t (&pk)[NW])
{
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        uint32_t v = 0;
#pragma unroll
        for (int i = 0; i < D8_PER; ++i) {
            const int d = id[i] - 3 * w;
            v += (id[i] >= 0 && d >= 0 && d < 3) ? (1u << (10 * d)) : 0u;
        }
        pk[w] = v;
    }
}

template <int NW>
__device__ __forceinline__ int d8_field(const uint32_t (&pk)[NW], int e)
{
    int r = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w)
        if (e / 3 == w) r = (pk[w] >> (10 * (e - 3 * w))) & 1023;
    return r;
}

template <int NW>
__global__ __launch_bounds__(D8_THREADS) void dispatch8_kernel(const int32_t* __restrict__ ids, int64_t A,
                                                              int E, int32_t* __restrict__ offsets,
                                                              int32_t* __restrict__ perm)
{
    __shared__ int wtot[D8_WAVES][64];   // per wave and expert, this chunk
    __shared__ int ebase[64];            // next position of each expert
    __shared__ int etot[64];             // whole-input counts (multi-chunk)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t nchunk = (A + D8_CHUNK - 1) / D8_CHUNK;
    if (nchunk == 0) {
        if (tid <= E) offsets[tid] = 0;
        return;
    }
    auto load = [&](int64_t c, int (&id)[D8_PER]) {
        const int64_t a0 = c * D8_CHUNK + (int64_t)tid * D8_PER;
#pragma unroll
        for (int i = 0; i < D8_PER; ++i) {
            // ids come from the router and lie in [0, E); the clamp keeps a
            // corrupted id from indexing past the histogram
            id[i] = a0 + i < A ? min(max(ids[a0 + i], 0), E - 1) : -1;
        }
    };
    // wave-inclusive prefix of the packed counts; wtot gets the wave totals
    auto wave_scan = [&](uint32_t (&pk)[NW]) {
#pragma unroll
        for (int w = 0; w < NW; ++w) {
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t v = __shfl_up(pk[w], o, 64);
                if (lane >= o) pk[w] += v;
            }
        }
        if (lane == 63) {
            for (int e = 0; e < E; ++e) wtot[wave][e] = d8_field<NW>(pk, e);
        }
    };
    int id[D8_PER];
    uint32_t pk[NW];
    if (nchunk > 1) {
        // counting pass: whole-input totals per expert
        if (tid < 64) etot[tid] = 0;
        for (int64_t c = 0; c < nchunk; ++c) {
            load(c, id);
            d8_pack<NW>(id, pk);
            wave_scan(pk);
            __syncthreads();
            if (tid < E) {
                int t = 0;
                for (int w = 0; w < D8_WAVES; ++w) t += wtot[w][tid];
                etot[tid] += t;
            }
            __syncthreads();
        }
    }
    for (int64_t c = 0; c < nchunk; ++c) {
        load(c, id);
        d8_pack<NW>(id, pk);
        uint32_t own[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) own[w] = pk[w];
        wave_scan(pk);
        __syncthreads();
        if (wave == 0) {
            // lane e: the chunk's count of expert e and the waves' exclusive bases
            int run = 0;
            if (lane < E) {
                for (int w = 0; w < D8_WAVES; ++w) {
                    const int t = wtot[w][lane];
                    wtot[w][lane] = run;
                    run += t;
                }
            }
            if (c == 0) {
                // expert offsets: exclusive scan of the whole-input counts
                const int cnt = lane < E ? (nchunk > 1 ? etot[lane] : run) : 0;
                int incl = cnt;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int v = __shfl_up(incl, o, 64);
                    if (lane >= o) incl += v;
                }
                if (lane < E) {
                    offsets[lane] = incl - cnt;
                    ebase[lane] = incl - cnt;
                }
                if (lane == E - 1) offsets[E] = incl;
            }
            // (wtot now holds the waves' bases; etot the chunk's counts,
            // added to ebase after the placement)
            if (lane < E) etot[lane] = run;
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < D8_PER; ++i) {
            const int e = id[i];
            if (e >= 0) {
                int r = 0;
#pragma unroll
                for (int i2 = 0; i2 < i; ++i2) r += id[i2] == e;
                const int pre = d8_field<NW>(pk, e) - d8_field<NW>(own, e);  // lanes before
                const int64_t a = c * D8_CHUNK + (int64_t)tid * D8_PER + i;
                perm[ebase[e] + wtot[wave][e] + pre + r] = static_cast<int32_t>(a);
            }
        }
        __syncthreads();
        if (tid < E) ebase[tid] += etot[tid];
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_router_topk(const bf16_t* x, const bf16_t* router_w, const float* bias,
                              int64_t T, int d, int E, int k, int32_t* topk_ids, float* topk_w,
                              float* logits, hipStream_t stream)
{
    if (T == 0) return hipSuccess;
    // From a few hundred tokens on (up to 16 experts) the matrix-core kernel:
    // it reads the router rows once per 16 tokens instead of once per token
    // (route + dispatch, Mixtral layer: 576 tokens 19.6 -> 14.5 us, 4096
    // tokens 41 -> 28 us); below that both take one memory round trip and
    // the per-token kernel spreads over more CUs.
    if (E <= 16 && T > 256) {
        const int64_t tiles = (T + 15) / 16;
        if (tiles > 0x7fffffff) return hipErrorInvalidValue;
        router_mfma_kernel<<<static_cast<unsigned>(tiles), RM_THREADS, 0, stream>>>(
            x, router_w, bias, T, d, E, k, topk_ids, topk_w, logits);
        return hipGetLastError();
    }
    // 64 / EMAX tokens per workgroup pass where that still makes 256
    // workgroups; fewer tokens, one per workgroup.  Measured on MI355X (route
    // + dispatch, E = 8): 4096 tokens 62 -> 42 us; 64 tokens 11.5 us with one
    // per workgroup, 16.8 us with eight.
    const int tpb = E <= 8 ? 8 : (E <= 16 ? 4 : (E <= 32 ? 2 : 1));
    const bool multi = T >= 256LL * tpb;
#define MOE_ROUTE(EMAX_, TPB_)                                                                    \
    {                                                                                             \
        const int64_t npass = (T + (TPB_) - 1) / (TPB_);                                          \
        const unsigned grid = static_cast<unsigned>(npass < 16384 ? npass : 16384);               \
        router_topk_kernel<EMAX_, TPB_><<<grid, ROUTE_THREADS, 0, stream>>>(                      \
            x, router_w, bias, T, d, E, k, topk_ids, topk_w, logits);                             \
    }
    if (E <= 8) {
        if (multi) MOE_ROUTE(8, 8) else MOE_ROUTE(8, 1)
    } else if (E <= 16) {
        if (multi) MOE_ROUTE(16, 4) else MOE_ROUTE(16, 1)
    } else if (E <= 32) {
        if (multi) MOE_ROUTE(32, 2) else MOE_ROUTE(32, 1)
    } else {
        MOE_ROUTE(64, 1)
    }
#undef MOE_ROUTE
    return hipGetLastError();
}

hipError_t launch_dispatch(const int32_t* topk_ids, int64_t A, int E, int32_t* offsets,
                           int32_t* perm, hipStream_t stream)
{
    // up to 1024 assignments (decode steps) the one-per-thread kernel, with
    // one chunk and no counting pass; above, 8 per thread (Mixtral layer,
    // 8192 assignments: route + dispatch 27.9 -> 19.3 us; 128 assignments:
    // 10.4-11.0 us one per thread, 12.0 us eight per thread)
    if (A <= DISPATCH_THREADS) {
        dispatch_kernel<<<1, DISPATCH_THREADS, 0, stream>>>(topk_ids, A, E, offsets, perm);
        return hipGetLastError();
    }
#define MOE_D8(NW_) dispatch8_kernel<NW_><<<1, D8_THREADS, 0, stream>>>(topk_ids, A, E, offsets, perm)
    if (E <= 9)
        MOE_D8(3);
    else if (E <= 18)
        MOE_D8(6);
    else
        MOE_D8(D8_MAXW);
#undef MOE_D8
    return hipGetLastError();
}

}  // namespace moe
