// Attention of one decode step over a paged KV cache, gfx950: the rotary
// position embedding of the new token's query and key, its key/value append
// to the cache, and grouped-query attention of every query head over its
// request's cached positions.
//
// Cache layout: [pages, Hkv, page, hd] bf16 for keys and values alike, so one
// page of one KV head (page * hd values) is contiguous.  Position s of the
// request of token t lives in page page_table[t * maxp + s / page], slot
// s % page.
//
// Decode attention is bound by reading the cache (2 * hd * 2 bytes per
// position and KV head): every cached byte is read once, and the query heads
// that share a KV head (the GQA group) are all served from that one read.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

namespace {

// One thread per (token, head, pair i < hd/2) over the Hq query, Hkv key and
// Hkv value heads of qkv [T, (Hq + 2 Hkv) hd] (f32 projections).  Query and
// key heads are rotated: element i pairs with i + hd/2, angle
// pos * theta^(-2i/hd), computed in double (positions reach tens of
// thousands, where a float angle would be off by ~1e-3 rad), then the pair is
// rotated in f32.  Queries go to q_out [T, Hq, hd]; keys and values into the
// cache at the token's position, all rounded to bf16.
__global__ __launch_bounds__(256) void rope_append_kernel(const float* qkv, const int32_t* pos,
                                                          const int32_t* page_table, int maxp,
                                                          int npages, int64_t T, int Hq, int Hkv,
                                                          int hd, int page, double theta,
                                                          bf16_t* q_out, bf16_t* kc, bf16_t* vc)
{
    const int half = hd / 2;
    const int nh = Hq + 2 * Hkv;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= T * nh * half) return;
    const int64_t t = idx / (nh * half);
    const int r = static_cast<int>(idx - t * nh * half);
    const int head = r / half, i = r - head * half;
    const int p = pos[t];
    const float* src = qkv + (t * nh + head) * hd;
    float a = src[i], b = src[i + half];
    if (head < Hq + Hkv) {
        double s, c;
        sincos(static_cast<double>(p) * pow(theta, -2.0 * i / hd), &s, &c);
        const float cf = static_cast<float>(c), sf = static_cast<float>(s);
        const float ra = a * cf - b * sf, rb = b * cf + a * sf;
        a = ra;
        b = rb;
    }
    bf16_t* dst;
    if (head < Hq) {
        dst = q_out + (t * Hq + head) * hd;
    } else {
        // a position or page outside the cache (invalid input) writes nothing
        if (p < 0 || p >= maxp * page) return;
        const int64_t pg = page_table[t * maxp + p / page];
        if (pg < 0 || pg >= npages) return;
        const bool key = head < Hq + Hkv;
        const int g = key ? head - Hq : head - Hq - Hkv;
        dst = (key ? kc : vc) + ((pg * Hkv + g) * page + p % page) * hd;
    }
    dst[i] = f32_to_bf16(a);
    dst[i + half] = f32_to_bf16(b);
}

constexpr int HD = 128;   // head dimension of these kernels
constexpr int LPP = 8;    // lanes per position: 16 dims each
constexpr int DPL = HD / LPP;
constexpr int PPB = 64 / LPP;  // positions per wave block
constexpr int NWAVE = 4;  // waves per workgroup
constexpr int MAXP = 4096;  // page-table entries per request held in LDS
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void widen16(const uint4& lo, const uint4& hi, float* f)
{
    const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        f[2 * j] = __uint_as_float(w[j] << 16);
        f[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
}

// Sum over an aligned group of 8 lanes, by DPP lane permutations (xor 1 and
// xor 2 within quads, then the mirror within the 8 lanes); every lane of the
// group ends with the sum.
template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL,
                                                                 0xF, 0xF, false));
}

__device__ __forceinline__ float sum8(float v)
{
    v += dpp<0xB1>(v);   // quad_perm [1, 0, 3, 2]
    v += dpp<0x4E>(v);   // quad_perm [2, 3, 0, 1]
    v += dpp<0x141>(v);  // row_half_mirror: quads 0 and 1 of each 8 lanes
    return v;
}

// One workgroup per (token t, KV head g); the GROUP query heads of g share
// every key/value read.  A wave takes blocks of 8 positions (8 lanes per
// position, 16 dims per lane) and keeps, per lane group, its own running max,
// sum and weighted value sum (online softmax in base 2: each score is
// multiplied by scale * log2(e)).  Query and key stay bf16 pairs: the dot
// products run as 2-wide bf16 dot instructions accumulating in f32 (half the
// instructions of widening both and multiplying in f32, and no registers for
// widened keys; measured 62-74 -> 60-68 us for 268 MB of cache).  The wave's
// blocks are loaded through a ring of NB register sets, NB - 1 blocks ahead
// of the one being multiplied.  The lane groups are merged by shuffles, the
// waves through LDS.
//
// With nsplit > 1 (few tokens, long contexts) the request's position blocks
// are cut into nsplit contiguous ranges, one workgroup each (workgroup
// (t, g, s) = blockIdx (t * Hkv + g) * nsplit + s); each writes its running
// max, sum and unnormalised weighted value sum to part [.., nsplit, GROUP,
// HD + 2] and attn_merge_kernel combines the ranges in order.
template <int GROUP>
__global__ __launch_bounds__(NWAVE * 64) void attn_decode_kernel(
    const bf16_t* q, const bf16_t* kc, const bf16_t* vc, const int32_t* page_table, int maxp,
    const int32_t* ctx, int npages, int Hq, int Hkv, int page, float scale, int nsplit,
    float* part, bf16_t* out)
{
    __shared__ float s_acc[NWAVE][GROUP][HD];
    __shared__ float s_ml[NWAVE][GROUP][2];
    __shared__ int s_page[MAXP];
    const int split = blockIdx.x % nsplit;
    const int tg = blockIdx.x / nsplit;
    const int t = tg / Hkv, g = tg - t * Hkv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int sub = lane & (LPP - 1), pp = lane / LPP;
    // a context outside [1, maxp * page] or a page id outside the cache
    // (invalid input) is clamped: no read leaves the cache
    const int L = min(max(ctx[t], 1), maxp * page);
    // the request's page ids, once, in LDS: a block's address then waits on
    // an LDS read, not on a memory load (memory loads retire in order, so
    // waiting for a page id would also wait for every key/value load before
    // it)
    const int npg = (L + page - 1) / page;
    for (int j = tid; j < npg; j += NWAVE * 64) {
        const int pg = page_table[(int64_t)t * maxp + j];
        s_page[j] = pg < 0 ? 0 : (pg >= npages ? npages - 1 : pg);
    }
    __syncthreads();
    const float qs = scale * 1.44269504088896340736f;  // scores in base 2

    uint32_t qb[GROUP][DPL / 2];  // the query's bf16 pairs (exact; the scale goes on the score)
#pragma unroll
    for (int h = 0; h < GROUP; ++h) {
        const bf16_t* qr = q + ((int64_t)t * Hq + g * GROUP + h) * HD + DPL * sub;
        const uint4 lo = ldg16(qr), hi = ldg16(qr + 8);
        qb[h][0] = lo.x; qb[h][1] = lo.y; qb[h][2] = lo.z; qb[h][3] = lo.w;
        qb[h][4] = hi.x; qb[h][5] = hi.y; qb[h][6] = hi.z; qb[h][7] = hi.w;
    }
    float m[GROUP], l[GROUP], acc[GROUP][DPL];
#pragma unroll
    for (int h = 0; h < GROUP; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.0f;
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[h][i] = 0.0f;
    }

    // this workgroup's blocks [bbeg, bend) of the request's position blocks
    const int nblk_all = (L + PPB - 1) / PPB;
    const int per = (nblk_all + nsplit - 1) / nsplit;
    const int bbeg = split * per;
    const int nblk = min(nblk_all, bbeg + per);  // blocks are numbered from 0; this range ends here
    auto addr = [&](int b) {
        int s = PPB * b + pp;
        s = s < L ? s : L - 1;  // dead positions read the last one (not used)
        const int64_t pg = s_page[s / page];
        return ((pg * Hkv + g) * page + s % page) * HD + DPL * sub;
    };
    auto update = [&](int b, const uint4* kv) {
        if (PPB * b + pp >= L) return;  // uniform over the lane group
        float vf[DPL];
        widen16(kv[2], kv[3], vf);
        const uint32_t kw[DPL / 2] = {kv[0].x, kv[0].y, kv[0].z, kv[0].w,
                                      kv[1].x, kv[1].y, kv[1].z, kv[1].w};
        float sd[GROUP];
#pragma unroll
        for (int h = 0; h < GROUP; ++h) {
            float d = 0.0f;
#pragma unroll
            for (int i = 0; i < DPL / 2; ++i)
                d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, qb[h][i]),
                                                    __builtin_bit_cast(bf16x2, kw[i]), d, false);
            sd[h] = d * qs;
        }
#pragma unroll
        for (int h = 0; h < GROUP; ++h) sd[h] = sum8(sd[h]);
#pragma unroll
        for (int h = 0; h < GROUP; ++h) {
            const float mn = fmaxf(m[h], sd[h]);
            const float cold = exp2f(m[h] - mn);  // 0 while nothing was seen (m = -inf)
            const float p = exp2f(sd[h] - mn);
            l[h] = fmaf(l[h], cold, p);
#pragma unroll
            for (int i = 0; i < DPL; ++i) acc[h][i] = fmaf(acc[h][i], cold, p * vf[i]);
            m[h] = mn;
        }
    };
    // blocks past the last are clamped to real positions (loaded, not used),
    // so every load is issued and the memory-counter waits stay static
    constexpr int NB = 3;
    uint4 ring[NB][4];
    auto load = [&](uint4* r, int b) {
        const int64_t o = addr(b < nblk ? b : nblk - 1);
        r[0] = ldg16(kc + o);
        r[1] = ldg16(kc + o + 8);
        r[2] = ldg16(vc + o);
        r[3] = ldg16(vc + o + 8);
    };
    if (bbeg < nblk) {
#pragma unroll
        for (int i = 0; i < NB - 1; ++i) load(ring[i], bbeg + wave + i * NWAVE);
    }
    for (int b0 = bbeg + wave; b0 < nblk; b0 += NB * NWAVE) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int b = b0 + i * NWAVE;
            if (b >= nblk) break;  // uniform over the wave
            load(ring[(i + NB - 1) % NB], b + (NB - 1) * NWAVE);
            update(b, ring[i]);
        }
    }

    // merge the lane groups of the wave (same dims, disjoint positions)
#pragma unroll
    for (int o = LPP; o < 64; o <<= 1) {
#pragma unroll
        for (int h = 0; h < GROUP; ++h) {
            const float mo = __shfl_xor(m[h], o, 64);
            const float lo = __shfl_xor(l[h], o, 64);
            const float mn = fmaxf(m[h], mo);
            const float ca = mn == -INFINITY ? 0.0f : exp2f(m[h] - mn);
            const float cb = mn == -INFINITY ? 0.0f : exp2f(mo - mn);
            l[h] = l[h] * ca + lo * cb;
#pragma unroll
            for (int i = 0; i < DPL; ++i) {
                const float ao = __shfl_xor(acc[h][i], o, 64);
                acc[h][i] = acc[h][i] * ca + ao * cb;
            }
            m[h] = mn;
        }
    }
    if (pp == 0) {
#pragma unroll
        for (int h = 0; h < GROUP; ++h) {
#pragma unroll
            for (int i = 0; i < DPL; ++i) s_acc[wave][h][DPL * sub + i] = acc[h][i];
            if (sub == 0) {
                s_ml[wave][h][0] = m[h];
                s_ml[wave][h][1] = l[h];
            }
        }
    }
    __syncthreads();
    // merge the waves and normalise (or hand the range's state over): one
    // thread per (head, dim)
    for (int j = tid; j < GROUP * HD; j += NWAVE * 64) {
        const int h = j / HD, dd = j - h * HD;
        float mt = -INFINITY;
#pragma unroll
        for (int w = 0; w < NWAVE; ++w) mt = fmaxf(mt, s_ml[w][h][0]);
        float lt = 0.0f, at = 0.0f;
        if (mt != -INFINITY) {  // -inf: an empty range (only with nsplit > 1)
#pragma unroll
            for (int w = 0; w < NWAVE; ++w) {
                const float c = exp2f(s_ml[w][h][0] - mt);  // an empty wave has m = -inf: 0
                lt = fmaf(s_ml[w][h][1], c, lt);
                at = fmaf(s_acc[w][h][dd], c, at);
            }
        }
        if (nsplit == 1) {
            out[((int64_t)t * Hq + g * GROUP + h) * HD + dd] = f32_to_bf16(at / lt);
        } else {
            float* pr = part + (((int64_t)tg * nsplit + split) * GROUP + h) * (HD + 2);
            pr[dd] = at;
            if (dd == 0) {
                pr[HD] = mt;
                pr[HD + 1] = lt;
            }
        }
    }
}

// Combines the nsplit ranges of attn_decode_kernel, in range order: one
// workgroup per (token, KV head), one thread per (head, dim).
template <int GROUP>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float* part, int nsplit, int Hq,
                                                         int Hkv, bf16_t* out)
{
    const int tg = blockIdx.x;
    const int t = tg / Hkv, g = tg - t * Hkv;
    for (int j = threadIdx.x; j < GROUP * HD; j += 256) {
        const int h = j / HD, dd = j - h * HD;
        const float* pr = part + ((int64_t)tg * nsplit * GROUP + h) * (HD + 2);
        const int64_t step = (int64_t)GROUP * (HD + 2);
        float mt = -INFINITY;
        for (int s = 0; s < nsplit; ++s) mt = fmaxf(mt, pr[s * step + HD]);
        float lt = 0.0f, at = 0.0f;
        for (int s = 0; s < nsplit; ++s) {
            const float c = exp2f(pr[s * step + HD] - mt);  // an empty range: m = -inf, 0
            lt = fmaf(pr[s * step + HD + 1], c, lt);
            at = fmaf(pr[s * step + dd], c, at);
        }
        out[((int64_t)t * Hq + g * GROUP + h) * HD + dd] = f32_to_bf16(at / lt);
    }
}

}  // namespace

bool attention_supported(int Hq, int Hkv, int hd, int page, int maxp)
{
    if (hd != HD || Hkv < 1 || Hq % Hkv || page < 8 || page % 8 || maxp > MAXP) return false;
    const int group = Hq / Hkv;
    return group == 1 || group == 2 || group == 4 || group == 8;
}

hipError_t launch_rope_append(const float* qkv, const int32_t* pos, const int32_t* page_table,
                              int maxp, int npages, int64_t T, int Hq, int Hkv, int hd, int page,
                              double theta, bf16_t* q_out, bf16_t* kc, bf16_t* vc,
                              hipStream_t stream)
{
    const int64_t n = T * (Hq + 2 * Hkv) * (hd / 2);
    const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
    rope_append_kernel<<<blocks, 256, 0, stream>>>(qkv, pos, page_table, maxp, npages, T, Hq, Hkv,
                                                   hd, page, theta, q_out, kc, vc);
    return hipGetLastError();
}

int attention_splits(int64_t T, int Hkv, int maxp, int page)
{
    // enough workgroups for every CU (two per CU), ranges of at least 256
    // positions, at most 32 ranges
    const int64_t base = T * Hkv;
    const int64_t want = (512 + base - 1) / base;
    const int64_t most = ((int64_t)maxp * page + 255) / 256;
    int64_t s = want < most ? want : most;
    s = s < 1 ? 1 : (s > 32 ? 32 : s);
    return static_cast<int>(s);
}

size_t attention_scratch_bytes(int64_t T, int Hq, int Hkv, int nsplit)
{
    return nsplit > 1 ? (size_t)T * Hkv * nsplit * (Hq / Hkv) * (HD + 2) * sizeof(float) : 0;
}

hipError_t launch_attention_decode(const bf16_t* q, const bf16_t* kc, const bf16_t* vc,
                                   const int32_t* page_table, int maxp, int npages,
                                   const int32_t* ctx, int64_t T, int Hq, int Hkv, int page,
                                   float scale, int nsplit, float* part, bf16_t* out,
                                   hipStream_t stream)
{
    const unsigned blocks = static_cast<unsigned>(T * Hkv * nsplit);
    const unsigned merge = static_cast<unsigned>(T * Hkv);
#define MOE_ATTN(GROUP_)                                                                          \
    attn_decode_kernel<GROUP_><<<blocks, NWAVE * 64, 0, stream>>>(q, kc, vc, page_table, maxp, ctx, \
                                                                  npages, Hq, Hkv, page, scale,   \
                                                                  nsplit, part, out);             \
    if (nsplit > 1) attn_merge_kernel<GROUP_><<<merge, 256, 0, stream>>>(part, nsplit, Hq, Hkv, out);
    switch (Hq / Hkv) {
    case 1: MOE_ATTN(1) break;
    case 2: MOE_ATTN(2) break;
    case 4: MOE_ATTN(4) break;
    default: MOE_ATTN(8) break;
    }
#undef MOE_ATTN
    return hipGetLastError();
}

}  // namespace moe
