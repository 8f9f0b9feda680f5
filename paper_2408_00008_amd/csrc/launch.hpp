// Host-side launchers of the gfx950 kernels.  Arguments are validated by the
// C ABI layer (api.cpp) before any of these is called; each launcher only
// enqueues work on `stream` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

typedef uint16_t bf16_t;

// Router GEMM (f32) + top-k + softmax over the selected logits, one token per
// workgroup slot.  logits may be null.
hipError_t launch_router_topk(const bf16_t* x, const bf16_t* router_w, const float* bias,
                              int64_t T, int d, int E, int k, int32_t* topk_ids, float* topk_w,
                              float* logits, hipStream_t stream);

// Expert histogram, exclusive scan and the stable expert-major permutation.
hipError_t launch_dispatch(const int32_t* topk_ids, int64_t A, int E, int32_t* offsets,
                           int32_t* perm, hipStream_t stream);

hipError_t launch_permute(const bf16_t* x, const int32_t* perm, int64_t A, int d, int k,
                          bf16_t* x_perm, hipStream_t stream);

// nslices (device int, null = 1, clamped to [1, max_slices]): y holds that
// many partial-sum slices of [T*k, d], summed per slot in ascending order
hipError_t launch_combine(const float* y, const float* residual, int64_t T, int d, int k,
                          bf16_t* out, float* out_f32, hipStream_t stream,
                          const int* nslices = nullptr, int max_slices = 1);

// Folds the reduction-part slices of the experts with at least mlo rows into
// slice 0 (y [smax, A, d] f32) after launch_tiled_down(mlo, ksplit_max =
// smax) ran with grid tiled_down_grid and nk = ffn / 64 reduction steps; the
// part count is recomputed on the device.  *parts_out (may be null) = 1.
hipError_t launch_fold_parts(float* y, int64_t A, int d, const int32_t* offsets, int E, int mlo,
                             const int32_t* perm, int nk, int per_xcd, int smax, int* parts_out,
                             hipStream_t stream);

// *p = v, stream-ordered (a kernel, so it may be captured into a graph)
hipError_t launch_fill_i32(int32_t* p, int32_t v, hipStream_t stream);

hipError_t launch_rmsnorm(const float* h, const bf16_t* gamma, int64_t T, int d, float eps,
                          bf16_t* a, hipStream_t stream);

// Decode attention (attention.hip): RoPE of the new token's query/key heads
// and the key/value append to the paged cache; grouped-query attention over
// the cache.  Cache layout [pages, Hkv, page, hd] bf16.
bool attention_supported(int Hq, int Hkv, int hd, int page, int maxp);
hipError_t launch_rope_append(const float* qkv, const int32_t* pos, const int32_t* page_table,
                              int maxp, int npages, int64_t T, int Hq, int Hkv, int hd, int page,
                              double theta, bf16_t* q_out, bf16_t* kc, bf16_t* vc,
                              hipStream_t stream);
// Position ranges per (token, KV head) so that the grid fills the GPU (few
// tokens, long contexts); the partial states need attention_scratch_bytes.
int attention_splits(int64_t T, int Hkv, int maxp, int page);
size_t attention_scratch_bytes(int64_t T, int Hq, int Hkv, int nsplit);
hipError_t launch_attention_decode(const bf16_t* q, const bf16_t* kc, const bf16_t* vc,
                                   const int32_t* page_table, int maxp, int npages,
                                   const int32_t* ctx, int64_t T, int Hq, int Hkv, int page,
                                   float scale, int nsplit, float* part, bf16_t* out,
                                   hipStream_t stream);

// Expert GEMMs.  `rows_hint` = T*k (an upper bound of any expert's rows) picks
// the tile shape; the real per-expert row counts are read on the device.
struct UpArgs {
    const bf16_t* x;         // token rows: x[gather ? gather[r]/kslots : r]
    const int32_t* gather;   // null = identity
    int kslots;
    const int32_t* offsets;  // [E+1]
    const bf16_t* w1;        // [E,ffn,d]
    const bf16_t* w3;        // [E,ffn,d]
    bf16_t* h;               // [A,ffn]
    int64_t A;
    int d, ffn, E;
    // 8-bit weights (then w1/w3 are unused): E4M3 bytes [E,ffn,d] and per-row
    // scales [E,ffn]
    const uint8_t* q1 = nullptr;
    const float* s1 = nullptr;
    const uint8_t* q3 = nullptr;
    const float* s3 = nullptr;
    // only experts with mlo <= rows <= mhi (the others are another launch's)
    int mlo = 0, mhi = 0x7fffffff;
    // streaming kernels: 16-row token groups per pass (0 = by rows per expert)
    int groups = 0;
    // streaming kernels: top-k expert of each assignment [A] (A <=
    // kStreamListMax); the kernel builds the offsets and the row order from
    // it, and offsets / gather are not read
    const int32_t* ids = nullptr;
};

struct DownArgs {
    const bf16_t* h;         // [A,ffn]
    const int32_t* offsets;  // [E+1]
    const bf16_t* w2;        // [E,d,ffn]
    const float* topk_w;     // [A] or null
    const int32_t* perm;     // [A] or null
    float* y;                // [A,d]
    int64_t A;
    int d, ffn, E;
    // 8-bit weights (then w2 is unused): E4M3 bytes [E,d,ffn], scales [E,d]
    const uint8_t* q2 = nullptr;
    const float* s2 = nullptr;
    int mlo = 0, mhi = 0x7fffffff;
    int groups = 0;
    // tiled kernel: y has room for ksplit_max slices [A,d]; the kernel picks
    // how many reduction parts to use (1 = y only) and stores that count to
    // *ksplit_out (device int, may be null)
    int ksplit_max = 1;
    int* ksplit_out = nullptr;
    // streaming kernels: as in UpArgs (offsets / perm are then not read)
    const int32_t* ids = nullptr;
};

// Assignments up to which the streaming kernels keep the routing tables in
// LDS (and can build them from the top-k ids).
constexpr int kStreamListMax = 1024;

enum GemmVariant { VARIANT_AUTO = 0, VARIANT_STREAM = 1, VARIANT_TILED = 2 };

// Supplies `bytes` of 256-byte aligned device scratch for one forward call,
// or returns an error status (with its message set).
typedef int (*ScratchFn)(size_t bytes, void** out);

// Chooses the kernel family for these sizes (resolves VARIANT_AUTO).
int resolve_variant(int requested, int64_t A, int E);

hipError_t launch_up(const UpArgs& a, int variant, hipStream_t stream);
hipError_t launch_down(const DownArgs& a, int variant, hipStream_t stream);

}  // namespace moe
