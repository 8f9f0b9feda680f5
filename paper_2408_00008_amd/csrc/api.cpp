// C ABI of libmoe: argument validation, scratch management and kernel
// sequencing.  Every check runs before the first HIP call, so a rejected call
// enqueues nothing and touches no device state.
#include "moe.h"

#include <hip/hip_runtime.h>

#include <atomic>
#include <cerrno>
#include <cstdint>
#include <cstdlib>
#include <cstdarg>
#include <cstdio>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>
#include <string>
#include <unordered_map>

#include "launch.hpp"

namespace moe {
hipError_t launch_stream_up(const UpArgs& a, int64_t rows_max, hipStream_t stream);
hipError_t launch_stream_down(const DownArgs& a, int64_t rows_max, hipStream_t stream);
hipError_t launch_tiled_up(const UpArgs& a, hipStream_t stream);
hipError_t launch_tiled_down(const DownArgs& a, hipStream_t stream);
int tiled_down_grid(const DownArgs& a);
bool tiled_supported(int d, int ffn, int64_t rows);
}  // namespace moe

namespace {

thread_local std::string g_last_error;
std::atomic<int> g_variant{moe::VARIANT_AUTO};

moe_status_t fail(moe_status_t s, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

moe_status_t ok()
{
    g_last_error.clear();
    return MOE_OK;
}

moe_status_t hip_fail(hipError_t e, const char* what)
{
    return fail(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Range {
    const void* p;
    size_t bytes;
};

bool overlap(Range a, Range b)
{
    if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
    return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

constexpr int kMaxE = 64, kMaxK = 8, kMaxDim = 65536;

moe_status_t check_T(int64_t T, int32_t k)
{
    if (T < 0) return fail(MOE_ERR_INVALID_ARG, "T=%lld must be >= 0", (long long)T);
    if (k >= 1 && T * (int64_t)k >= (int64_t(1) << 31))
        return fail(MOE_ERR_UNSUPPORTED, "T*k=%lld must be < 2^31", (long long)(T * k));
    return MOE_OK;
}

moe_status_t check_Ek(int32_t E, int32_t k)
{
    if (E < 1) return fail(MOE_ERR_INVALID_ARG, "E=%d must be >= 1", E);
    if (E > kMaxE) return fail(MOE_ERR_UNSUPPORTED, "E=%d exceeds %d", E, kMaxE);
    if (k < 1) return fail(MOE_ERR_INVALID_ARG, "k=%d must be >= 1", k);
    if (k > E) return fail(MOE_ERR_INVALID_ARG, "k=%d exceeds E=%d", k, E);
    if (k > kMaxK) return fail(MOE_ERR_UNSUPPORTED, "k=%d exceeds %d", k, kMaxK);
    return MOE_OK;
}

// the expert-GEMM stages: E counts the experts whose weights are passed, which
// may be a shard of the routed experts, so k is not bounded by it
moe_status_t check_Ek_stage(int32_t E, int32_t k)
{
    if (E < 1) return fail(MOE_ERR_INVALID_ARG, "E=%d must be >= 1", E);
    if (E > kMaxE) return fail(MOE_ERR_UNSUPPORTED, "E=%d exceeds %d", E, kMaxE);
    if (k < 1) return fail(MOE_ERR_INVALID_ARG, "k=%d must be >= 1", k);
    if (k > kMaxK) return fail(MOE_ERR_UNSUPPORTED, "k=%d exceeds %d", k, kMaxK);
    return MOE_OK;
}

moe_status_t check_dim(const char* name, int32_t v)
{
    if (v < 1) return fail(MOE_ERR_INVALID_ARG, "%s=%d must be >= 1", name, v);
    if (v % 64 != 0) return fail(MOE_ERR_UNSUPPORTED, "%s=%d must be a multiple of 64", name, v);
    if (v > kMaxDim) return fail(MOE_ERR_UNSUPPORTED, "%s=%d exceeds %d", name, v, kMaxDim);
    return MOE_OK;
}

#define TRY(expr)                      \
    do {                               \
        moe_status_t s_ = (expr);      \
        if (s_ != MOE_OK) return s_;   \
    } while (0)

moe_status_t need(const void* p, const char* name)
{
    if (!p) return fail(MOE_ERR_INVALID_ARG, "%s is NULL", name);
    if (!aligned16(p)) return fail(MOE_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return MOE_OK;
}

moe_status_t maybe(const void* p, const char* name)
{
    if (p && !aligned16(p)) return fail(MOE_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return MOE_OK;
}

// a buffer whose size scales with T: may be NULL when T == 0
moe_status_t need_rows(const void* p, const char* name, int64_t T)
{
    return T == 0 ? maybe(p, name) : need(p, name);
}

moe_status_t no_overlap(const char* oname, Range o, std::initializer_list<std::pair<const char*, Range>> ins)
{
    for (const auto& in : ins)
        if (overlap(o, in.second))
            return fail(MOE_ERR_INVALID_ARG, "%s overlaps %s", oname, in.first);
    return MOE_OK;
}

// ---- workspace ------------------------------------------------------------

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Reduction parts the tiled down GEMM may use inside moe_forward: 1, 2 or 4,
// each part at least 8 steps of 64 (the kernel picks the count on the
// device from the real tile count).  Only where the tiled kernel runs by
// default and the tiles fill fewer than 16 rounds of 256 workgroups, where a
// cut evens out the last round.
// Largest power of two <= requested, <= 16 and leaving each part at least 8
// reduction steps of 64.
int parts_cap(int32_t ffn, int requested)
{
    const int steps = ffn / 64;
    int c = 1;
    while (c * 2 <= requested && c * 2 <= 16 && steps / (c * 2) >= 8) c *= 2;
    return c;
}

// An expert with more rows than this takes its own launch in the streaming
// regime (see run_up / run_down).
constexpr int64_t kLightRows = 64;

// Reduction parts moe_forward's down GEMM may use (the slices of y):
//  * tiled regime (over 64 rows per expert on average): up to 4, where the
//    tiles fill fewer than 16 rounds of 256 workgroups;
//  * streaming regime with T > kLightRows, where an expert may be heavy: up to
//    2 for the heavy experts' tiled launch, which runs next to the light
//    experts' streaming launch (the parts are folded back into slice 0
//    before the combine).  Measured on MI355X, one expert of 194 rows and
//    seven of 45, down + combine: 264 us with the heavy expert streaming in
//    64-row passes after the light ones; side by side 224 / 233 / 242 / 242 us
//    with at most 2 / 4 / 8 / 16 parts (in sequence 8 parts were best: the
//    fewer the parts, the fewer CUs the heavy launch takes from the light).
int down_split_max(int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k)
{
    const int64_t A = T * k;
    if (!moe::tiled_supported(d, ffn, A)) return 1;
    if (A <= 64LL * E) return T > kLightRows ? parts_cap(ffn, 2) : 1;
    const int64_t items = (int64_t)(d / 256) * (A / 256 + E);
    if (items >= 16 * 256) return 1;
    return parts_cap(ffn, 4);
}

struct Layout {
    size_t ids, w, off, perm, h, y, ns, total;
    int nsplit;  // slices of y
};

Layout layout(int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k)
{
    const size_t A = static_cast<size_t>(T) * k;
    Layout L{};
    L.nsplit = down_split_max(T, d, ffn, E, k);
    size_t o = 0;
    L.ids = o;  o += align256(A * 4);
    L.w = o;    o += align256(A * 4);
    L.off = o;  o += align256(static_cast<size_t>(E + 1) * 4);
    L.perm = o; o += align256(A * 4);
    L.h = o;    o += align256(A * static_cast<size_t>(ffn) * 2);
    L.y = o;    o += align256(A * static_cast<size_t>(d) * 4 * L.nsplit);
    L.ns = o;   o += 256;
    L.total = o;
    return L;
}

struct DeviceScratch {
    void* ptr = nullptr;
    size_t bytes = 0;
    // the buffer was handed to a call made while its stream was being
    // captured: a graph may still replay with it, so a growth keeps it alive
    // (retired) instead of freeing it
    bool captured = false;
};
std::mutex g_ws_mu;
// per device: slot 0 serves moe_forward / moe_forward_ex, slot 1 the
// partial states of moe_attention_decode
std::unordered_map<int, DeviceScratch> g_ws[2];
// per device: buffers replaced while a captured graph may still use them;
// freed by moe_release_workspace only
std::unordered_map<int, std::vector<void*>> g_retired;

// Cap on each library-owned scratch buffer, in bytes, from the environment
// variable MOE_WORKSPACE_LIMIT_BYTES (read on every call; unset or empty = no
// cap).  A call that needs more returns MOE_ERR_NO_MEMORY before any HIP call.
moe_status_t workspace_limit(size_t* limit)
{
    *limit = SIZE_MAX;
    const char* s = std::getenv("MOE_WORKSPACE_LIMIT_BYTES");
    if (!s || !*s) return MOE_OK;
    char* end = nullptr;
    errno = 0;
    const unsigned long long v = std::strtoull(s, &end, 10);
    if (end == s || *end != '\0' || errno == ERANGE || s[0] == '-')
        return fail(MOE_ERR_INVALID_ARG, "MOE_WORKSPACE_LIMIT_BYTES='%s' is not a byte count", s);
    *limit = static_cast<size_t>(v);
    return MOE_OK;
}

moe_status_t library_workspace(size_t need_bytes, hipStream_t stream, void** out, int slot = 0)
{
    size_t limit = SIZE_MAX;
    TRY(workspace_limit(&limit));
    if (need_bytes > limit)
        return fail(MOE_ERR_NO_MEMORY,
                    "library scratch of %zu bytes needed, above MOE_WORKSPACE_LIMIT_BYTES=%zu "
                    "(pass a caller workspace to moe_forward_ex instead)",
                    need_bytes, limit);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    e = hipStreamIsCapturing(stream, &cs);
    if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
    std::lock_guard<std::mutex> lk(g_ws_mu);
    DeviceScratch& s = g_ws[slot][dev];
    if (s.bytes < need_bytes) {
        if (cs != hipStreamCaptureStatusNone)
            return fail(MOE_ERR_NO_MEMORY,
                        "library scratch must grow to %zu bytes while the stream is being "
                        "captured; call once outside capture first",
                        need_bytes);
        if (s.ptr) {
            if (s.captured) {
                g_retired[dev].push_back(s.ptr);
            } else {
                // earlier work on any stream may still use the old buffer
                e = hipDeviceSynchronize();
                if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
                (void)hipFree(s.ptr);
            }
            s.ptr = nullptr;
            s.bytes = 0;
            s.captured = false;
        }
        size_t grow = need_bytes + need_bytes / 4;
        if (grow > limit) grow = limit;
        e = hipMalloc(&s.ptr, grow);
        if (e != hipSuccess) {
            s.ptr = nullptr;
            return fail(MOE_ERR_NO_MEMORY, "hipMalloc(%zu) failed: %s", grow, hipGetErrorString(e));
        }
        s.bytes = grow;
    }
    if (cs != hipStreamCaptureStatusNone) s.captured = true;
    *out = s.ptr;
    return MOE_OK;
}

int64_t rows_bound(int64_t T, int32_t) { return T; }

// Expert weights of one call: bf16 matrices, or E4M3 bytes with per-row f32
// scales (q*, s* non-NULL).
struct ExpertWeights {
    const moe_bf16_t* w1 = nullptr;
    const moe_bf16_t* w3 = nullptr;
    const moe_bf16_t* w2 = nullptr;
    const uint8_t* q1 = nullptr;
    const float* s1 = nullptr;
    const uint8_t* q3 = nullptr;
    const float* s3 = nullptr;
    const uint8_t* q2 = nullptr;
    const float* s2 = nullptr;
    bool f8 = false;
    bool fp8() const { return f8; }
};

moe_status_t check_up_weights(const ExpertWeights& w)
{
    if (!w.fp8()) {
        TRY(need(w.w1, "w1"));
        return need(w.w3, "w3");
    }
    TRY(need(w.q1, "w1q"));
    TRY(need(w.s1, "w1s"));
    TRY(need(w.q3, "w3q"));
    return need(w.s3, "w3s");
}

moe_status_t check_down_weights(const ExpertWeights& w)
{
    if (!w.fp8()) return need(w.w2, "w2");
    TRY(need(w.q2, "w2q"));
    return need(w.s2, "w2s");
}

// (name, range) of every weight buffer of an up or down call
std::vector<std::pair<const char*, Range>> weight_ranges(const ExpertWeights& w, int32_t d,
                                                         int32_t ffn, int32_t E, bool up, bool down)
{
    const size_t n = (size_t)E * ffn * d;
    std::vector<std::pair<const char*, Range>> r;
    if (!w.fp8()) {
        if (up) r.push_back({"w1", {w.w1, n * 2}}), r.push_back({"w3", {w.w3, n * 2}});
        if (down) r.push_back({"w2", {w.w2, n * 2}});
    } else {
        if (up) {
            r.push_back({"w1q", {w.q1, n}});
            r.push_back({"w1s", {w.s1, (size_t)E * ffn * 4}});
            r.push_back({"w3q", {w.q3, n}});
            r.push_back({"w3s", {w.s3, (size_t)E * ffn * 4}});
        }
        if (down) {
            r.push_back({"w2q", {w.q2, n}});
            r.push_back({"w2s", {w.s2, (size_t)E * d * 4}});
        }
    }
    return r;
}

moe_status_t no_overlap_v(const char* oname, Range o, const std::vector<std::pair<const char*, Range>>& ins)
{
    for (const auto& in : ins)
        if (overlap(o, in.second))
            return fail(MOE_ERR_INVALID_ARG, "%s overlaps %s", oname, in.first);
    return MOE_OK;
}

// Per-expert kernel choice.  Rows per expert are known only on the device, so
// when a call of the streaming regime may hold experts of very different
// sizes (more than kLightRows tokens, e.g. a skewed decode step), each expert
// GEMM becomes two launches that each keep the experts of their size class:
// experts with at most kLightRows rows stream their weights in one pass;
// heavier ones take the tiled kernel (up, bf16 or 8-bit weights) or, for the
// down GEMM, the streaming kernel with 128-row passes.  Measured on MI355X
// with one expert of 194 rows and seven of 45 (T = 256): up 426 -> 392 us,
// down 261 -> 228 us.  Where the caller provides slices for reduction parts
// (moe_forward, moe_swiglu_down_parts), the heavy down GEMM takes the tiled
// kernel too, its reduction cut into up to 16 parts, folded into slice 0.

// ---- expert groups side by side -------------------------------------------
//
// In a split launch the light experts stream their weights (HBM-bound, on
// every CU) while the heavy experts' tiled launch is MFMA-bound on at most a
// few hundred workgroups; on two streams they overlap.  Measured on MI355X,
// skewed T = 256 up GEMM: 397 us in sequence, 373 us side by side with the
// light launch enqueued first (388 us heavy first).  The side stream is per
// device (default priority, created on first use, kept until the process
// ends); fork and join are event waits, so the caller's stream sees one
// ordered operation.  While the caller's stream is being captured into a
// graph the two launches run in sequence on it.
struct SideStream {
    hipStream_t s = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
    std::mutex mu;  // one fork/join at a time: the two events are reused
};
std::mutex g_side_mu;
std::unordered_map<int, SideStream*> g_side;  // null: could not be created

SideStream* side_stream()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    std::lock_guard<std::mutex> lk(g_side_mu);
    auto it = g_side.find(dev);
    if (it != g_side.end()) return it->second;
    SideStream* ss = new SideStream;
    if (hipStreamCreateWithFlags(&ss->s, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&ss->fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&ss->join, hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();
        ss = nullptr;  // the launches then run in sequence
    }
    g_side[dev] = ss;
    return ss;
}

// side = false: the two launches run in sequence on `stream` (callers that
// must not create the side stream's resources)
template <class Light, class Heavy>
hipError_t run_side_by_side(hipStream_t stream, Light light, Heavy heavy, bool side = true)
{
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(stream, &cs);
    if (e != hipSuccess) return e;
    SideStream* ss = (side && cs == hipStreamCaptureStatusNone) ? side_stream() : nullptr;
    if (!ss) {
        e = light(stream);
        return e != hipSuccess ? e : heavy(stream);
    }
    std::lock_guard<std::mutex> lk(ss->mu);
    if ((e = hipEventRecord(ss->fork, stream)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(ss->s, ss->fork, 0)) != hipSuccess) return e;
    const hipError_t el = light(stream);
    const hipError_t eh = el == hipSuccess ? heavy(ss->s) : hipSuccess;
    // join after a failed launch too: whatever the side stream took on stays
    // ordered before the caller's later work
    e = hipEventRecord(ss->join, ss->s);
    if (e == hipSuccess) e = hipStreamWaitEvent(stream, ss->join, 0);
    return el != hipSuccess ? el : (eh != hipSuccess ? eh : e);
}

bool split_by_rows(int64_t rows_max, int64_t A, int E)
{
    return g_variant.load() == moe::VARIANT_AUTO && rows_max > kLightRows &&
           moe::resolve_variant(moe::VARIANT_AUTO, A, E) == moe::VARIANT_STREAM;
}

hipError_t run_up(const moe::UpArgs& a, int64_t T, hipStream_t stream, bool side = true)
{
    const int64_t rmax = rows_bound(T, a.kslots);
    // routing from the top-k ids exists on the streaming kernel only
    if (a.ids) return moe::launch_stream_up(a, rmax, stream);
    const bool tiled_ok = moe::tiled_supported(a.d, a.ffn, a.A);
    if (split_by_rows(rmax, a.A, a.E)) {
        moe::UpArgs light = a, heavy = a;
        light.mhi = kLightRows;
        heavy.mlo = kLightRows + 1;
        if (tiled_ok)
            return run_side_by_side(
                stream, [&](hipStream_t s) { return moe::launch_stream_up(light, kLightRows, s); },
                [&](hipStream_t s) { return moe::launch_tiled_up(heavy, s); }, side);
        hipError_t e = moe::launch_stream_up(light, kLightRows, stream);
        if (e != hipSuccess) return e;
        heavy.groups = 8;
        return moe::launch_stream_up(heavy, rmax, stream);
    }
    const int v = moe::resolve_variant(g_variant.load(), a.A, a.E);
    if (v == moe::VARIANT_TILED && tiled_ok) return moe::launch_tiled_up(a, stream);
    return moe::launch_stream_up(a, rmax, stream);
}

// With a.ksplit_out set, y has room for a.ksplit_max slices [A,d] and on
// return *a.ksplit_out (stream-ordered) holds how many of them the combine
// must sum; *sliced tells whether that may exceed 1.
hipError_t run_down(const moe::DownArgs& a, int64_t T, int32_t k, hipStream_t stream,
                    bool* sliced = nullptr, bool side = true)
{
    if (sliced) *sliced = false;
    const bool parts = a.ksplit_out != nullptr;
    auto uncut = [&](hipError_t e) {
        if (e != hipSuccess || !parts) return e;
        return moe::launch_fill_i32(a.ksplit_out, 1, stream);
    };
    const int64_t rmax = rows_bound(T, k);
    if (a.ids) return uncut(moe::launch_stream_down(a, rmax, stream));
    if (split_by_rows(rmax, a.A, a.E)) {
        moe::DownArgs light = a, heavy = a;
        light.mhi = kLightRows;
        light.ksplit_out = nullptr;
        heavy.mlo = kLightRows + 1;
        if (parts && a.ksplit_max > 1 && moe::tiled_supported(a.d, a.ffn, a.A)) {
            // the fold recomputes the part count and sets *ksplit_out = 1
            heavy.ksplit_out = nullptr;
            return run_side_by_side(
                stream, [&](hipStream_t s) { return moe::launch_stream_down(light, kLightRows, s); },
                [&](hipStream_t s) {
                    hipError_t e = moe::launch_tiled_down(heavy, s);
                    if (e != hipSuccess) return e;
                    return moe::launch_fold_parts(a.y, a.A, a.d, a.offsets, a.E, heavy.mlo,
                                                  a.topk_w ? a.perm : nullptr, a.ffn / 64,
                                                  moe::tiled_down_grid(heavy) / 8, a.ksplit_max,
                                                  a.ksplit_out, s);
                },
                side);
        }
        hipError_t e = moe::launch_stream_down(light, kLightRows, stream);
        if (e != hipSuccess) return e;
        heavy.groups = 8;
        heavy.ksplit_out = nullptr;
        return uncut(moe::launch_stream_down(heavy, rmax, stream));
    }
    const int v = moe::resolve_variant(g_variant.load(), a.A, a.E);
    if (v == moe::VARIANT_TILED && moe::tiled_supported(a.d, a.ffn, a.A)) {
        if (sliced) *sliced = parts;
        return moe::launch_tiled_down(a, stream);
    }
    return uncut(moe::launch_stream_down(a, rmax, stream));
}

}  // namespace

namespace moe {
int resolve_variant(int requested, int64_t A, int E)
{
    if (requested == VARIANT_STREAM || requested == VARIANT_TILED) return requested;
    // weight streaming while an expert's rows are few: up to 64 rows per
    // expert on average (measured on MI355X: streaming ahead at 64, the tiled
    // kernel from 96)
    return (A <= 64LL * E) ? VARIANT_STREAM : VARIANT_TILED;
}
}  // namespace moe

namespace {

// ---- entry points shared by the bf16 and the 8-bit weight formats --------

moe_status_t swiglu_up_impl(const moe_bf16_t* x_perm, const int32_t* perm,
                            const int32_t* expert_offsets, const ExpertWeights& w, int64_t T,
                            int32_t d, int32_t ffn, int32_t E, int32_t k, moe_bf16_t* h,
                            hipStream_t stream)
{
    TRY(check_Ek_stage(E, k));
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(check_dim("ffn", ffn));
    TRY(need_rows(x_perm, "x_perm", T));
    TRY(need(expert_offsets, "expert_offsets"));
    TRY(check_up_weights(w));
    TRY(need_rows(h, "h", T));
    TRY(maybe(perm, "perm"));
    const size_t A = static_cast<size_t>(T) * k;
    const size_t xrows = perm ? static_cast<size_t>(T) : A;
    auto ins = weight_ranges(w, d, ffn, E, true, false);
    ins.push_back({"x", {x_perm, xrows * d * 2}});
    ins.push_back({"expert_offsets", {expert_offsets, (size_t)(E + 1) * 4}});
    ins.push_back({"perm", {perm, A * 4}});
    TRY(no_overlap_v("h", {h, A * ffn * 2}, ins));
    if (T == 0) return ok();
    moe::UpArgs a{x_perm, perm, k, expert_offsets, w.w1, w.w3, h, (int64_t)A, d, ffn, E};
    a.q1 = w.q1, a.s1 = w.s1, a.q3 = w.q3, a.s3 = w.s3;
    hipError_t e = run_up(a, T, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "expert up kernel launch");
}

// max_parts > 1 with parts != null: y holds max_parts slices [A,d] for the
// reduction parts of the tiled kernel, their count stored to *parts
moe_status_t swiglu_down_impl(const moe_bf16_t* h, const int32_t* expert_offsets,
                              const ExpertWeights& w, const float* topk_w, const int32_t* perm,
                              int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k, float* y,
                              hipStream_t stream, int max_parts = 1, int32_t* parts = nullptr)
{
    TRY(check_Ek_stage(E, k));
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(check_dim("ffn", ffn));
    TRY(need_rows(h, "h", T));
    TRY(need(expert_offsets, "expert_offsets"));
    TRY(check_down_weights(w));
    TRY(maybe(topk_w, "topk_w"));
    TRY(maybe(perm, "perm"));
    TRY(need_rows(y, "y", T));
    const size_t A = static_cast<size_t>(T) * k;
    auto ins = weight_ranges(w, d, ffn, E, false, true);
    ins.push_back({"h", {h, A * ffn * 2}});
    ins.push_back({"topk_w", {topk_w, A * 4}});
    ins.push_back({"perm", {perm, A * 4}});
    ins.push_back({"expert_offsets", {expert_offsets, (size_t)(E + 1) * 4}});
    const size_t ybytes = A * d * 4 * static_cast<size_t>(max_parts);
    if (parts) {
        ins.push_back({"y", {y, ybytes}});
        TRY(no_overlap_v("parts", {parts, 4}, ins));
        ins.pop_back();
    }
    TRY(no_overlap_v("y", {y, ybytes}, ins));
    if (T == 0) {
        if (!parts) return ok();
        hipError_t e = moe::launch_fill_i32(parts, 1, stream);
        return e == hipSuccess ? ok() : hip_fail(e, "fill kernel launch");
    }
    const bool scatter = topk_w && perm;
    moe::DownArgs a{h, expert_offsets, w.w2, scatter ? topk_w : nullptr, scatter ? perm : nullptr,
                    y, (int64_t)A, d, ffn, E};
    a.q2 = w.q2, a.s2 = w.s2;
    a.ksplit_max = parts ? parts_cap(ffn, max_parts) : 1;
    a.ksplit_out = parts;
    hipError_t e = run_down(a, T, k, stream);
    if (e != hipSuccess) return hip_fail(e, "expert down kernel launch");
    return ok();
}

// scratch_fn (optional): supplies the scratch when workspace is NULL instead
// of the library-owned buffer; the split launches then run in sequence on
// `stream` (no side stream is created)
moe_status_t forward_impl(const moe_bf16_t* x, const moe_bf16_t* router_w,
                          const float* router_bias, const ExpertWeights& w, int64_t T, int32_t d,
                          int32_t ffn, int32_t E, int32_t k, const float* residual,
                          moe_bf16_t* out, float* out_f32, void* workspace,
                          size_t workspace_bytes, hipStream_t stream,
                          moe::ScratchFn scratch_fn = nullptr)
{
    TRY(check_Ek(E, k));
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(check_dim("ffn", ffn));
    TRY(need_rows(x, "x", T));
    TRY(need(router_w, "router_w"));
    TRY(maybe(router_bias, "router_bias"));
    TRY(check_up_weights(w));
    TRY(check_down_weights(w));
    TRY(maybe(residual, "residual"));
    TRY(maybe(out, "out"));
    TRY(maybe(out_f32, "out_f32"));
    if (!out && !out_f32 && T > 0)
        return fail(MOE_ERR_INVALID_ARG, "out and out_f32 are both NULL");
    if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return fail(MOE_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
    const size_t td = static_cast<size_t>(T) * d;
    auto ins = weight_ranges(w, d, ffn, E, true, true);
    ins.push_back({"x", {x, td * 2}});
    ins.push_back({"router_w", {router_w, (size_t)E * d * 2}});
    ins.push_back({"router_bias", {router_bias, (size_t)E * 4}});
    TRY(no_overlap_v("out", {out, td * 2}, ins));
    TRY(no_overlap("out", {out, td * 2}, {{"residual", {residual, td * 4}}, {"out_f32", {out_f32, td * 4}}}));
    TRY(no_overlap_v("out_f32", {out_f32, td * 4}, ins));
    if (residual && out_f32 != residual)
        TRY(no_overlap("out_f32", {out_f32, td * 4}, {{"residual", {residual, td * 4}}}));
    const Layout L = layout(T, d, ffn, E, k);
    if (workspace && workspace_bytes < L.total)
        return fail(MOE_ERR_NO_MEMORY, "workspace of %zu bytes is smaller than the %zu needed",
                    workspace_bytes, L.total);
    if (workspace) {
        const Range ws{workspace, L.total};
        TRY(no_overlap_v("workspace", ws, ins));
        TRY(no_overlap("workspace", ws, {{"out", {out, td * 2}}, {"out_f32", {out_f32, td * 4}},
                       {"residual", {residual, td * 4}}}));
    }
    if (T == 0) return ok();

    void* base = workspace;
    if (!base) {
        if (scratch_fn)
            TRY(static_cast<moe_status_t>(scratch_fn(L.total, &base)));
        else
            TRY(library_workspace(L.total, stream, &base));
    }
    const bool side = scratch_fn == nullptr;
    char* b = static_cast<char*>(base);
    int32_t* ids = reinterpret_cast<int32_t*>(b + L.ids);
    float* gw = reinterpret_cast<float*>(b + L.w);
    int32_t* offs = reinterpret_cast<int32_t*>(b + L.off);
    int32_t* perm = reinterpret_cast<int32_t*>(b + L.perm);
    moe::bf16_t* h = reinterpret_cast<moe::bf16_t*>(b + L.h);
    float* y = reinterpret_cast<float*>(b + L.y);
    const int64_t A = T * k;

    hipError_t e = moe::launch_router_topk(x, router_w, router_bias, T, d, E, k, ids, gw, nullptr,
                                           stream);
    if (e != hipSuccess) return hip_fail(e, "router kernel launch");
    // Both GEMMs on the streaming kernels and few assignments: each of their
    // workgroups builds the expert offsets and row order from the top-k ids
    // in LDS, and no dispatch kernel runs.
    const bool by_ids = A <= moe::kStreamListMax && !split_by_rows(rows_bound(T, k), A, E) &&
                        moe::resolve_variant(g_variant.load(), A, E) == moe::VARIANT_STREAM;
    if (!by_ids) {
        e = moe::launch_dispatch(ids, A, E, offs, perm, stream);
        if (e != hipSuccess) return hip_fail(e, "dispatch kernel launch");
    }
    moe::UpArgs ua{x, perm, k, offs, w.w1, w.w3, h, A, d, ffn, E};
    ua.q1 = w.q1, ua.s1 = w.s1, ua.q3 = w.q3, ua.s3 = w.s3;
    if (by_ids) {
        ua.ids = ids;
        ua.gather = nullptr;
        ua.offsets = nullptr;
    }
    e = run_up(ua, T, stream, side);
    if (e != hipSuccess) return hip_fail(e, "expert up kernel launch");
    moe::DownArgs da{h, offs, w.w2, gw, perm, y, A, d, ffn, E};
    da.q2 = w.q2, da.s2 = w.s2;
    if (by_ids) {
        da.ids = ids;
        da.perm = nullptr;
        da.offsets = nullptr;
    }
    da.ksplit_max = L.nsplit;
    // the part count is only needed (and only written) where y has slices
    da.ksplit_out = L.nsplit > 1 ? reinterpret_cast<int*>(b + L.ns) : nullptr;
    bool sliced = false;
    e = run_down(da, T, k, stream, &sliced, side);
    if (e != hipSuccess) return hip_fail(e, "expert down kernel launch");
    e = moe::launch_combine(y, residual, T, d, k, out, out_f32, stream,
                            sliced ? da.ksplit_out : nullptr, L.nsplit);
    if (e != hipSuccess) return hip_fail(e, "combine kernel launch");
    return ok();
}

ExpertWeights bf16_weights(const moe_bf16_t* w1, const moe_bf16_t* w3, const moe_bf16_t* w2)
{
    ExpertWeights w;
    w.w1 = w1, w.w3 = w3, w.w2 = w2;
    return w;
}

// the format is fixed by the entry point, not by which pointers are NULL, so
// a NULL byte array is reported as such
ExpertWeights fp8_weights(const uint8_t* q1, const float* s1, const uint8_t* q3, const float* s3,
                          const uint8_t* q2, const float* s2)
{
    ExpertWeights w;
    w.q1 = q1, w.s1 = s1, w.q3 = q3, w.s3 = s3, w.q2 = q2, w.s2 = s2;
    w.f8 = true;
    return w;
}

}  // namespace

namespace moe {
moe_status_t set_last_error(moe_status_t s, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

moe_status_t forward_fixed_scratch(const moe_bf16_t* x, const moe_bf16_t* router_w,
                                   const float* router_bias, const moe_bf16_t* w1,
                                   const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T,
                                   int32_t d, int32_t ffn, int32_t E, int32_t k,
                                   const float* residual, moe_bf16_t* out, float* out_f32,
                                   hipStream_t stream, ScratchFn scratch_fn)
{
    return forward_impl(x, router_w, router_bias, bf16_weights(w1, w3, w2), T, d, ffn, E, k,
                        residual, out, out_f32, nullptr, 0, stream, scratch_fn);
}
}  // namespace moe

namespace {
constexpr int kMaxHeads = 256, kMaxHd = 1024;

moe_status_t check_heads(int32_t Hq, int32_t Hkv, int32_t hd)
{
    if (Hq < 1 || Hkv < 1 || Hq % Hkv)
        return fail(MOE_ERR_INVALID_ARG, "Hq=%d must be a positive multiple of Hkv=%d", Hq, Hkv);
    if (Hq > kMaxHeads) return fail(MOE_ERR_UNSUPPORTED, "Hq=%d exceeds %d", Hq, kMaxHeads);
    if (hd < 2 || hd % 2 || hd > kMaxHd)
        return fail(MOE_ERR_INVALID_ARG, "hd=%d must be even, 2..%d", hd, kMaxHd);
    return MOE_OK;
}

moe_status_t check_cache(int32_t page, int32_t maxp, int64_t npages)
{
    if (page < 1 || maxp < 1 || npages < 1)
        return fail(MOE_ERR_INVALID_ARG, "page=%d, maxp=%d, npages=%lld must be >= 1", page, maxp,
                    (long long)npages);
    if ((int64_t)page * maxp >= (int64_t(1) << 31) || npages >= (int64_t(1) << 31))
        return fail(MOE_ERR_UNSUPPORTED, "cache geometry too large");
    return MOE_OK;
}
}  // namespace

namespace {
moe_status_t combine_impl(const float* y, const int32_t* parts, int32_t max_parts,
                          const float* residual, int64_t T, int32_t d, int32_t k,
                          moe_bf16_t* out, float* out_f32, hipStream_t stream)
{
    if (k < 1 || k > kMaxK) return fail(k < 1 ? MOE_ERR_INVALID_ARG : MOE_ERR_UNSUPPORTED,
                                        "k=%d out of range", k);
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(need_rows(y, "y", T));
    TRY(maybe(residual, "residual"));
    TRY(maybe(out, "out"));
    TRY(maybe(out_f32, "out_f32"));
    if (!out && !out_f32 && T > 0)
        return fail(MOE_ERR_INVALID_ARG, "out and out_f32 are both NULL");
    const size_t A = static_cast<size_t>(T) * k;
    const size_t td = static_cast<size_t>(T) * d;
    const size_t yb = A * d * 4 * static_cast<size_t>(max_parts);
    TRY(no_overlap("out", {out, td * 2}, {{"y", {y, yb}}, {"residual", {residual, td * 4}},
                   {"out_f32", {out_f32, td * 4}}, {"parts", {parts, 4}}}));
    if (out_f32 != residual)
        TRY(no_overlap("out_f32", {out_f32, td * 4}, {{"y", {y, yb}}, {"residual", {residual, td * 4}},
                       {"parts", {parts, 4}}}));
    else
        TRY(no_overlap("out_f32", {out_f32, td * 4}, {{"y", {y, yb}}, {"parts", {parts, 4}}}));
    if (T == 0) return ok();
    hipError_t e = moe::launch_combine(y, residual, T, d, k, out, out_f32, stream, parts, max_parts);
    return e == hipSuccess ? ok() : hip_fail(e, "combine kernel launch");
}
}  // namespace

extern "C" {

moe_status_t moe_route(const moe_bf16_t* x, const moe_bf16_t* router_w, const float* router_bias,
                       int64_t T, int32_t d, int32_t E, int32_t k, int32_t* topk_ids,
                       float* topk_w, int32_t* expert_offsets, int32_t* perm, float* logits,
                       hipStream_t stream)
{
    TRY(check_Ek(E, k));
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(need_rows(x, "x", T));
    TRY(need(router_w, "router_w"));
    TRY(maybe(router_bias, "router_bias"));
    TRY(need_rows(topk_ids, "topk_ids", T));
    TRY(need_rows(topk_w, "topk_w", T));
    TRY(need(expert_offsets, "expert_offsets"));
    TRY(need_rows(perm, "perm", T));
    TRY(maybe(logits, "logits"));
    const size_t A = static_cast<size_t>(T) * k;
    TRY(no_overlap("topk_ids", {topk_ids, A * 4}, {{"topk_w", {topk_w, A * 4}}, {"perm", {perm, A * 4}},
                   {"expert_offsets", {expert_offsets, (size_t)(E + 1) * 4}}}));
    TRY(no_overlap("perm", {perm, A * 4}, {{"topk_w", {topk_w, A * 4}},
                   {"expert_offsets", {expert_offsets, (size_t)(E + 1) * 4}}}));
    if (T == 0) return ok();
    hipError_t e = moe::launch_router_topk(x, router_w, router_bias, T, d, E, k, topk_ids, topk_w,
                                           logits, stream);
    if (e != hipSuccess) return hip_fail(e, "router kernel launch");
    e = moe::launch_dispatch(topk_ids, static_cast<int64_t>(A), E, expert_offsets, perm, stream);
    if (e != hipSuccess) return hip_fail(e, "dispatch kernel launch");
    return ok();
}

moe_status_t moe_permute(const moe_bf16_t* x, const int32_t* perm, int64_t T, int32_t d,
                         int32_t k, moe_bf16_t* x_perm, hipStream_t stream)
{
    if (k < 1 || k > kMaxK) return fail(k < 1 ? MOE_ERR_INVALID_ARG : MOE_ERR_UNSUPPORTED,
                                        "k=%d out of range", k);
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(need_rows(x, "x", T));
    TRY(need_rows(perm, "perm", T));
    TRY(need_rows(x_perm, "x_perm", T));
    const size_t A = static_cast<size_t>(T) * k;
    TRY(no_overlap("x_perm", {x_perm, A * d * 2}, {{"x", {x, (size_t)T * d * 2}}, {"perm", {perm, A * 4}}}));
    if (T == 0) return ok();
    hipError_t e = moe::launch_permute(x, perm, static_cast<int64_t>(A), d, k, x_perm, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "permute kernel launch");
}

moe_status_t moe_swiglu_up(const moe_bf16_t* x_perm, const int32_t* perm,
                           const int32_t* expert_offsets, const moe_bf16_t* w1,
                           const moe_bf16_t* w3, int64_t T, int32_t d, int32_t ffn, int32_t E,
                           int32_t k, moe_bf16_t* h, hipStream_t stream)
{
    return swiglu_up_impl(x_perm, perm, expert_offsets, bf16_weights(w1, w3, nullptr), T, d, ffn,
                          E, k, h, stream);
}

moe_status_t moe_swiglu_down(const moe_bf16_t* h, const int32_t* expert_offsets,
                             const moe_bf16_t* w2, const float* topk_w, const int32_t* perm,
                             int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k, float* y,
                             hipStream_t stream)
{
    return swiglu_down_impl(h, expert_offsets, bf16_weights(nullptr, nullptr, w2), topk_w, perm,
                            T, d, ffn, E, k, y, stream);
}

moe_status_t moe_swiglu_down_parts(const moe_bf16_t* h, const int32_t* expert_offsets,
                                   const moe_bf16_t* w2, const float* topk_w, const int32_t* perm,
                                   int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k,
                                   int32_t max_parts, float* y, int32_t* parts,
                                   hipStream_t stream)
{
    if (max_parts < 1) return fail(MOE_ERR_INVALID_ARG, "max_parts=%d must be >= 1", max_parts);
    if (!parts) return fail(MOE_ERR_INVALID_ARG, "parts is NULL");
    if (reinterpret_cast<uintptr_t>(parts) & 3u)
        return fail(MOE_ERR_INVALID_ARG, "parts is not 4-byte aligned");
    // the slices the caller sized y for; the kernel uses at most parts_cap of them
    return swiglu_down_impl(h, expert_offsets, bf16_weights(nullptr, nullptr, w2), topk_w, perm,
                            T, d, ffn, E, k, y, stream, max_parts, parts);
}

moe_status_t moe_swiglu_up_fp8(const moe_bf16_t* x_perm, const int32_t* perm,
                               const int32_t* expert_offsets, const uint8_t* w1q,
                               const float* w1s, const uint8_t* w3q, const float* w3s, int64_t T,
                               int32_t d, int32_t ffn, int32_t E, int32_t k, moe_bf16_t* h,
                               hipStream_t stream)
{
    return swiglu_up_impl(x_perm, perm, expert_offsets,
                          fp8_weights(w1q, w1s, w3q, w3s, nullptr, nullptr), T, d, ffn, E, k, h,
                          stream);
}

moe_status_t moe_swiglu_down_fp8(const moe_bf16_t* h, const int32_t* expert_offsets,
                                 const uint8_t* w2q, const float* w2s, const float* topk_w,
                                 const int32_t* perm, int64_t T, int32_t d, int32_t ffn, int32_t E,
                                 int32_t k, float* y, hipStream_t stream)
{
    return swiglu_down_impl(h, expert_offsets,
                            fp8_weights(nullptr, nullptr, nullptr, nullptr, w2q, w2s), topk_w,
                            perm, T, d, ffn, E, k, y, stream);
}

moe_status_t moe_swiglu_down_parts_fp8(const moe_bf16_t* h, const int32_t* expert_offsets,
                                       const uint8_t* w2q, const float* w2s, const float* topk_w,
                                       const int32_t* perm, int64_t T, int32_t d, int32_t ffn,
                                       int32_t E, int32_t k, int32_t max_parts, float* y,
                                       int32_t* parts, hipStream_t stream)
{
    if (max_parts < 1) return fail(MOE_ERR_INVALID_ARG, "max_parts=%d must be >= 1", max_parts);
    if (!parts) return fail(MOE_ERR_INVALID_ARG, "parts is NULL");
    if (reinterpret_cast<uintptr_t>(parts) & 3u)
        return fail(MOE_ERR_INVALID_ARG, "parts is not 4-byte aligned");
    return swiglu_down_impl(h, expert_offsets,
                            fp8_weights(nullptr, nullptr, nullptr, nullptr, w2q, w2s), topk_w,
                            perm, T, d, ffn, E, k, y, stream, max_parts, parts);
}

moe_status_t moe_grouped_swiglu(const moe_bf16_t* x_perm, const int32_t* expert_offsets,
                                const moe_bf16_t* w1, const moe_bf16_t* w3,
                                const moe_bf16_t* w2, const float* topk_w, const int32_t* perm,
                                int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k,
                                moe_bf16_t* h_ws, float* y, hipStream_t stream)
{
    TRY(check_Ek_stage(E, k));
    TRY(check_T(T, k));
    TRY(check_dim("d", d));
    TRY(check_dim("ffn", ffn));
    TRY(need(w2, "w2"));
    TRY(need_rows(y, "y", T));
    TRY(maybe(topk_w, "topk_w"));
    TRY(maybe(perm, "perm"));
    const size_t A = static_cast<size_t>(T) * k;
    TRY(no_overlap("y", {y, A * d * 4}, {{"h_ws", {h_ws, A * ffn * 2}}, {"x_perm", {x_perm, A * d * 2}}}));
    moe_status_t s =
        moe_swiglu_up(x_perm, nullptr, expert_offsets, w1, w3, T, d, ffn, E, k, h_ws, stream);
    if (s != MOE_OK) return s;
    return moe_swiglu_down(h_ws, expert_offsets, w2, topk_w, perm, T, d, ffn, E, k, y, stream);
}

moe_status_t moe_combine(const float* y, const float* residual, int64_t T, int32_t d, int32_t k,
                         moe_bf16_t* out, float* out_f32, hipStream_t stream)
{
    return combine_impl(y, nullptr, 1, residual, T, d, k, out, out_f32, stream);
}

moe_status_t moe_combine_parts(const float* y, const int32_t* parts, int32_t max_parts,
                               const float* residual, int64_t T, int32_t d, int32_t k,
                               moe_bf16_t* out, float* out_f32, hipStream_t stream)
{
    if (max_parts < 1) return fail(MOE_ERR_INVALID_ARG, "max_parts=%d must be >= 1", max_parts);
    if (!parts) return fail(MOE_ERR_INVALID_ARG, "parts is NULL");
    if (reinterpret_cast<uintptr_t>(parts) & 3u)
        return fail(MOE_ERR_INVALID_ARG, "parts is not 4-byte aligned");
    return combine_impl(y, parts, max_parts, residual, T, d, k, out, out_f32, stream);
}

size_t moe_workspace_size(int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k)
{
    if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E || k > kMaxK || d < 1 || ffn < 1 ||
        T * (int64_t)k >= (int64_t(1) << 31))
        return 0;
    return layout(T, d, ffn, E, k).total;
}

moe_status_t moe_forward_ex(const moe_bf16_t* x, const moe_bf16_t* router_w,
                            const float* router_bias, const moe_bf16_t* w1,
                            const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T, int32_t d,
                            int32_t ffn, int32_t E, int32_t k, const float* residual,
                            moe_bf16_t* out, float* out_f32, void* workspace,
                            size_t workspace_bytes, hipStream_t stream)
{
    return forward_impl(x, router_w, router_bias, bf16_weights(w1, w3, w2), T, d, ffn, E, k,
                        residual, out, out_f32, workspace, workspace_bytes, stream);
}

moe_status_t moe_forward_fp8_ex(const moe_bf16_t* x, const moe_bf16_t* router_w,
                                const float* router_bias, const uint8_t* w1q, const float* w1s,
                                const uint8_t* w3q, const float* w3s, const uint8_t* w2q,
                                const float* w2s, int64_t T, int32_t d, int32_t ffn, int32_t E,
                                int32_t k, const float* residual, moe_bf16_t* out,
                                float* out_f32, void* workspace, size_t workspace_bytes,
                                hipStream_t stream)
{
    return forward_impl(x, router_w, router_bias, fp8_weights(w1q, w1s, w3q, w3s, w2q, w2s), T, d,
                        ffn, E, k, residual, out, out_f32, workspace, workspace_bytes, stream);
}

moe_status_t moe_forward(const moe_bf16_t* x, const moe_bf16_t* router_w, const moe_bf16_t* w1,
                         const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T, int32_t d,
                         int32_t ffn, int32_t E, int32_t k, moe_bf16_t* out, hipStream_t stream)
{
    TRY(need_rows(out, "out", T));
    return moe_forward_ex(x, router_w, nullptr, w1, w3, w2, T, d, ffn, E, k, nullptr, out,
                          nullptr, nullptr, 0, stream);
}

moe_status_t moe_rmsnorm(const float* h, const moe_bf16_t* gamma, int64_t T, int32_t d, float eps,
                         moe_bf16_t* a, hipStream_t stream)
{
    if (T < 0) return fail(MOE_ERR_INVALID_ARG, "T=%lld must be >= 0", (long long)T);
    TRY(check_dim("d", d));
    if (!(eps >= 0.0f)) return fail(MOE_ERR_INVALID_ARG, "eps must be >= 0");
    TRY(need_rows(h, "h", T));
    TRY(need(gamma, "gamma"));
    TRY(need_rows(a, "a", T));
    const size_t td = static_cast<size_t>(T) * d;
    TRY(no_overlap("a", {a, td * 2}, {{"h", {h, td * 4}}, {"gamma", {gamma, (size_t)d * 2}}}));
    if (T == 0) return ok();
    hipError_t e = moe::launch_rmsnorm(h, gamma, T, d, eps, a, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "rmsnorm kernel launch");
}

moe_status_t moe_linear(const moe_bf16_t* x, const moe_bf16_t* w, int64_t T, int32_t K, int32_t N,
                        float* y, hipStream_t stream)
{
    TRY(check_T(T, 1));
    TRY(check_dim("K", K));
    TRY(check_dim("N", N));
    TRY(need_rows(x, "x", T));
    TRY(need(w, "w"));
    TRY(need_rows(y, "y", T));
    TRY(no_overlap("y", {y, (size_t)T * N * 4}, {{"x", {x, (size_t)T * K * 2}},
                   {"w", {w, (size_t)N * K * 2}}}));
    if (T == 0) return ok();
    // one matrix (offsets NULL): the tiled kernel where its 256 x 256 items
    // fill at least half the CUs of an MI355X, the weight-streaming kernel
    // below.  Measured, K = 4096, N = 6144: 2048 tokens 357 us streaming.
    moe::DownArgs a{x, nullptr, w, nullptr, nullptr, y, T, N, K, 1};
    const int64_t items = (int64_t)(N / 256) * ((T + 255) / 256);
    hipError_t e = (items >= 128 && moe::tiled_supported(N, K, T)) ? moe::launch_tiled_down(a, stream)
                                                                : moe::launch_stream_down(a, T, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "linear kernel launch");
}


moe_status_t moe_rope_kv_append(const float* qkv, const int32_t* pos, const int32_t* page_table,
                                int64_t T, int32_t Hq, int32_t Hkv, int32_t hd, int32_t page,
                                int32_t maxp, int64_t npages, double theta, moe_bf16_t* q_out,
                                moe_bf16_t* k_cache, moe_bf16_t* v_cache, hipStream_t stream)
{
    TRY(check_T(T, Hq + 2 * Hkv));
    TRY(check_heads(Hq, Hkv, hd));
    TRY(check_cache(page, maxp, npages));
    if (!(theta > 0.0) || !std::isfinite(theta)) return fail(MOE_ERR_INVALID_ARG, "theta must be > 0");
    TRY(need_rows(qkv, "qkv", T));
    TRY(need_rows(pos, "pos", T));
    TRY(need_rows(page_table, "page_table", T));
    TRY(need_rows(q_out, "q_out", T));
    TRY(need(k_cache, "k_cache"));
    TRY(need(v_cache, "v_cache"));
    const size_t cache = (size_t)npages * Hkv * page * hd * 2;
    const Range rk{k_cache, cache}, rv{v_cache, cache}, rq{q_out, (size_t)T * Hq * hd * 2};
    const std::initializer_list<std::pair<const char*, Range>> ins = {
        {"qkv", {qkv, (size_t)T * (Hq + 2 * Hkv) * hd * 4}}, {"pos", {pos, (size_t)T * 4}},
        {"page_table", {page_table, (size_t)T * maxp * 4}}};
    TRY(no_overlap("q_out", rq, ins));
    TRY(no_overlap("k_cache", rk, ins));
    TRY(no_overlap("v_cache", rv, ins));
    TRY(no_overlap("k_cache", rk, {{"v_cache", rv}, {"q_out", rq}}));
    TRY(no_overlap("v_cache", rv, {{"q_out", rq}}));
    if (T == 0) return ok();
    hipError_t e = moe::launch_rope_append(qkv, pos, page_table, maxp, static_cast<int>(npages), T,
                                           Hq, Hkv, hd, page, theta, q_out, k_cache, v_cache,
                                           stream);
    return e == hipSuccess ? ok() : hip_fail(e, "rope/append kernel launch");
}

moe_status_t moe_attention_decode(const moe_bf16_t* q, const moe_bf16_t* k_cache,
                                  const moe_bf16_t* v_cache, const int32_t* page_table,
                                  const int32_t* ctx, int64_t T, int32_t Hq, int32_t Hkv,
                                  int32_t hd, int32_t page, int32_t maxp, int64_t npages,
                                  float scale, moe_bf16_t* out, hipStream_t stream)
{
    TRY(check_T(T, Hkv));
    TRY(check_heads(Hq, Hkv, hd));
    TRY(check_cache(page, maxp, npages));
    if (!moe::attention_supported(Hq, Hkv, hd, page, maxp))
        return fail(MOE_ERR_UNSUPPORTED,
                    "attention needs hd = 128, Hq/Hkv in {1, 2, 4, 8}, page a multiple of 8 and "
                    "maxp <= 4096 (got hd=%d, Hq=%d, Hkv=%d, page=%d, maxp=%d)", hd, Hq, Hkv, page,
                    maxp);
    if (!(scale > 0.0f) || !std::isfinite(scale)) return fail(MOE_ERR_INVALID_ARG, "scale must be > 0");
    TRY(need_rows(q, "q", T));
    TRY(need(k_cache, "k_cache"));
    TRY(need(v_cache, "v_cache"));
    TRY(need_rows(page_table, "page_table", T));
    TRY(need_rows(ctx, "ctx", T));
    TRY(need_rows(out, "out", T));
    const size_t cache = (size_t)npages * Hkv * page * hd * 2;
    TRY(no_overlap("out", {out, (size_t)T * Hq * hd * 2},
                   {{"q", {q, (size_t)T * Hq * hd * 2}}, {"k_cache", {k_cache, cache}},
                    {"v_cache", {v_cache, cache}}, {"page_table", {page_table, (size_t)T * maxp * 4}},
                    {"ctx", {ctx, (size_t)T * 4}}}));
    if (T == 0) return ok();
    const int nsplit = moe::attention_splits(T, Hkv, maxp, page);
    void* part = nullptr;
    const size_t pbytes = moe::attention_scratch_bytes(T, Hq, Hkv, nsplit);
    if (pbytes) TRY(library_workspace(pbytes, stream, &part, 1));
    hipError_t e = moe::launch_attention_decode(q, k_cache, v_cache, page_table, maxp,
                                                static_cast<int>(npages), ctx, T, Hq, Hkv, page,
                                                scale, nsplit, static_cast<float*>(part), out,
                                                stream);
    return e == hipSuccess ? ok() : hip_fail(e, "attention kernel launch");
}

moe_status_t moe_release_workspace(void)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_ws_mu);
    e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    for (auto& slot : g_ws) {
        auto it = slot.find(dev);
        if (it == slot.end()) continue;
        if (it->second.ptr) (void)hipFree(it->second.ptr);
        slot.erase(it);
    }
    auto rt = g_retired.find(dev);
    if (rt != g_retired.end()) {
        for (void* p : rt->second) (void)hipFree(p);
        g_retired.erase(rt);
    }
    return ok();
}

int moe_gemm_variant_for(int64_t T, int32_t d, int32_t ffn, int32_t E, int32_t k)
{
    if (moe_workspace_size(T, d, ffn, E, k) == 0 || d % 64 || ffn % 64) return 0;
    if (split_by_rows(rows_bound(T, k), T * k, E)) return 3;
    const int v = moe::resolve_variant(g_variant.load(), T * k, E);
    return (v == moe::VARIANT_TILED && moe::tiled_supported(d, ffn, T * k)) ? moe::VARIANT_TILED
                                                                     : moe::VARIANT_STREAM;
}

int moe_set_gemm_variant(int variant)
{
    if (variant < moe::VARIANT_AUTO || variant > moe::VARIANT_TILED) return -1;
    return g_variant.exchange(variant);
}

const char* moe_status_string(int status)
{
    switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_NO_MEMORY: return "MOE_ERR_NO_MEMORY";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
    default: return "MOE_ERR_UNKNOWN";
    }
}

const char* moe_last_error(void) { return g_last_error.c_str(); }

int moe_version(void) { return 100; }

}  // extern "C"
