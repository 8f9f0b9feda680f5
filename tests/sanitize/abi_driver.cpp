// Drives the argument validation of every libmoe entry point (api.cpp) for a
// build with AddressSanitizer and UndefinedBehaviorSanitizer.  Every call
// here is rejected by validation, is empty (T = 0) or hits the scratch cap,
// so no kernel is launched and no device is needed: pointers are fake,
// 16-byte aligned device addresses that are never dereferenced on the host.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "moe.h"

namespace {

int g_fail = 0, g_checks = 0;

void expect(int got, int want, const char* what, const char* msg_part = nullptr)
{
    ++g_checks;
    const char* msg = moe_last_error();
    if (got != want || (msg_part && !std::strstr(msg, msg_part))) {
        std::fprintf(stderr, "FAIL %s: status %d (want %d), message '%s'\n", what, got, want, msg);
        ++g_fail;
    }
}

template <class T>
T* fake(uint64_t slot)
{
    return reinterpret_cast<T*>(uintptr_t((slot + 1) << 40));
}

}  // namespace

int main()
{
    using bf = moe_bf16_t;
    const bf* x = fake<bf>(0);
    const bf* rw = fake<bf>(1);
    const bf* w1 = fake<bf>(2);
    const bf* w3 = fake<bf>(3);
    const bf* w2 = fake<bf>(4);
    bf* out = fake<bf>(5);
    int32_t* ids = fake<int32_t>(6);
    float* gw = fake<float>(7);
    int32_t* offs = fake<int32_t>(8);
    int32_t* perm = fake<int32_t>(9);
    float* y = fake<float>(10);
    bf* h = fake<bf>(11);
    float* res = fake<float>(12);
    int32_t* parts = fake<int32_t>(13);
    const uint8_t* q = fake<uint8_t>(14);
    const float* sc = fake<float>(15);
    void* ws = fake<void>(16);

    // moe_forward: limits, pointers, aliasing, T = 0
    expect(moe_forward(x, rw, w1, w3, w2, 4, 128, 256, 65, 2, out, nullptr), MOE_ERR_UNSUPPORTED, "E=65");
    expect(moe_forward(x, rw, w1, w3, w2, 4, 128, 256, 8, 0, out, nullptr), MOE_ERR_INVALID_ARG, "k=0");
    expect(moe_forward(x, rw, w1, w3, w2, 4, 100, 256, 8, 2, out, nullptr), MOE_ERR_UNSUPPORTED, "d=100");
    expect(moe_forward(x, rw, w1, w3, w2, -1, 128, 256, 8, 2, out, nullptr), MOE_ERR_INVALID_ARG, "T<0");
    expect(moe_forward(x, rw, w1, w3, w2, int64_t(1) << 30, 128, 256, 8, 2, out, nullptr),
           MOE_ERR_UNSUPPORTED, "T*k", "2^31");
    expect(moe_forward(nullptr, rw, w1, w3, w2, 4, 128, 256, 8, 2, out, nullptr), MOE_ERR_INVALID_ARG,
           "x null", "x is NULL");
    expect(moe_forward(reinterpret_cast<const bf*>(uintptr_t(x) + 2), rw, w1, w3, w2, 4, 128, 256, 8,
                       2, out, nullptr), MOE_ERR_INVALID_ARG, "x misaligned", "aligned");
    expect(moe_forward(x, rw, w1, w3, w2, 4, 128, 256, 8, 2, const_cast<bf*>(x), nullptr),
           MOE_ERR_INVALID_ARG, "out aliases x", "overlaps");
    expect(moe_forward(x, rw, w1, w3, w2, 0, 128, 256, 8, 2, out, nullptr), MOE_OK, "T=0");
    // moe_forward_ex: workspace checks
    const size_t need = moe_workspace_size(4, 128, 256, 8, 2);
    expect(need > 0 ? MOE_OK : MOE_ERR_INVALID_ARG, MOE_OK, "workspace size");
    expect(moe_forward_ex(x, rw, nullptr, w1, w3, w2, 4, 128, 256, 8, 2, nullptr, out, nullptr,
                          static_cast<char*>(ws) + 16, need, nullptr),
           MOE_ERR_INVALID_ARG, "ws misaligned", "256-byte");
    expect(moe_forward_ex(x, rw, nullptr, w1, w3, w2, 4, 128, 256, 8, 2, nullptr, out, nullptr, ws,
                          need - 1, nullptr), MOE_ERR_NO_MEMORY, "ws small", "smaller than");
    expect(moe_forward_ex(x, rw, nullptr, w1, w3, w2, 4, 128, 256, 8, 2, nullptr, nullptr, nullptr,
                          ws, need, nullptr), MOE_ERR_INVALID_ARG, "no output", "both NULL");
    expect(moe_forward_ex(x, rw, nullptr, w1, w3, w2, 4, 128, 256, 8, 2, res, out, res,
                          reinterpret_cast<char*>(res) + 256, need, nullptr),
           MOE_ERR_INVALID_ARG, "ws overlaps residual", "workspace overlaps");
    // the library scratch cap: after validation, before any HIP call
    setenv("MOE_WORKSPACE_LIMIT_BYTES", "1000", 1);
    expect(moe_forward(x, rw, w1, w3, w2, 4, 128, 256, 8, 2, out, nullptr), MOE_ERR_NO_MEMORY, "cap",
           "MOE_WORKSPACE_LIMIT_BYTES");
    setenv("MOE_WORKSPACE_LIMIT_BYTES", "12x", 1);
    expect(moe_forward(x, rw, w1, w3, w2, 4, 128, 256, 8, 2, out, nullptr), MOE_ERR_INVALID_ARG,
           "cap unparsable", "not a byte count");
    unsetenv("MOE_WORKSPACE_LIMIT_BYTES");

    // routing, permutation, expert stages, combine
    expect(moe_route(x, rw, nullptr, 4, 128, 2, 3, ids, gw, offs, perm, nullptr, nullptr),
           MOE_ERR_INVALID_ARG, "route k>E");
    expect(moe_route(x, rw, nullptr, 4, 128, 8, 2, ids, reinterpret_cast<float*>(ids), offs, perm,
                     nullptr, nullptr), MOE_ERR_INVALID_ARG, "route overlap", "overlaps");
    expect(moe_route(x, rw, nullptr, 0, 128, 8, 2, ids, gw, offs, perm, nullptr, nullptr), MOE_OK,
           "route T=0");
    expect(moe_permute(x, perm, 4, 128, 2, const_cast<bf*>(x), nullptr), MOE_ERR_INVALID_ARG,
           "permute in place");
    expect(moe_swiglu_up(x, nullptr, offs, w1, w3, 4, 128, 256, 8, 2, const_cast<bf*>(w1), nullptr),
           MOE_ERR_INVALID_ARG, "up h overlaps w1", "overlaps w1");
    expect(moe_swiglu_down(h, offs, w2, gw, perm, 4, 128, 256, 8, 9, y, nullptr), MOE_ERR_UNSUPPORTED,
           "down k=9");
    expect(moe_swiglu_down_parts(h, offs, w2, gw, perm, 4, 128, 256, 8, 2, 0, y, parts, nullptr),
           MOE_ERR_INVALID_ARG, "parts max 0", "max_parts");
    expect(moe_swiglu_down_parts(h, offs, w2, gw, perm, 4, 128, 256, 8, 2, 2, y, nullptr, nullptr),
           MOE_ERR_INVALID_ARG, "parts null", "parts is NULL");
    expect(moe_grouped_swiglu(x, offs, w1, w3, w2, gw, perm, 4, 128, 256, 8, 2, h,
                              reinterpret_cast<float*>(h), nullptr), MOE_ERR_INVALID_ARG,
           "grouped y overlaps h");
    expect(moe_combine(y, nullptr, 4, 128, 2, nullptr, nullptr, nullptr), MOE_ERR_INVALID_ARG,
           "combine no output");
    expect(moe_combine_parts(y, parts, 0, nullptr, 4, 128, 2, out, nullptr, nullptr),
           MOE_ERR_INVALID_ARG, "combine parts max 0");
    expect(moe_rmsnorm(y, w1, 4, 128, -1.0f, out, nullptr), MOE_ERR_INVALID_ARG, "rmsnorm eps");

    // 8-bit weights
    expect(moe_swiglu_up_fp8(x, nullptr, offs, nullptr, sc, q, sc, 4, 128, 256, 8, 2, h, nullptr),
           MOE_ERR_INVALID_ARG, "fp8 up null", "w1q is NULL");
    expect(moe_swiglu_down_fp8(h, offs, q, nullptr, gw, perm, 4, 128, 256, 8, 2, y, nullptr),
           MOE_ERR_INVALID_ARG, "fp8 down null scale", "w2s is NULL");
    expect(moe_forward_fp8_ex(x, rw, nullptr, q, sc, q, sc, q, sc, 4, 128, 256, 8, 2, nullptr,
                              const_cast<bf*>(reinterpret_cast<const bf*>(q)), nullptr, nullptr, 0,
                              nullptr), MOE_ERR_INVALID_ARG, "fp8 out overlaps w1q", "overlaps");
    expect(moe_swiglu_down_parts_fp8(h, offs, q, sc, gw, perm, 4, 128, 256, 8, 2, 0, y, parts,
                                     nullptr), MOE_ERR_INVALID_ARG, "fp8 parts max 0");

    // decoder-layer calls
    expect(moe_linear(x, w1, 4, 100, 64, y, nullptr), MOE_ERR_UNSUPPORTED, "linear K=100");
    expect(moe_rope_kv_append(y, ids, perm, 4, 32, 8, 128, 16, 4, 64, -1.0, out,
                              const_cast<bf*>(w1), const_cast<bf*>(w2), nullptr),
           MOE_ERR_INVALID_ARG, "rope theta");
    expect(moe_attention_decode(x, w1, w2, perm, ids, 4, 32, 8, 64, 16, 4, 64, 0.1f, out, nullptr),
           MOE_ERR_UNSUPPORTED, "attention hd=64");
    expect(moe_attention_decode(x, w1, w2, perm, ids, 4, 32, 8, 128, 16, 4, 64, -0.1f, out, nullptr),
           MOE_ERR_INVALID_ARG, "attention scale");

    // host-only queries
    expect(moe_workspace_size(4, 128, 256, 8, 9) == 0 ? MOE_OK : 1, MOE_OK, "workspace size k=9");
    expect(moe_gemm_variant_for(64, 4096, 14336, 8, 2), 1, "variant decode");
    expect(moe_gemm_variant_for(4096, 4096, 14336, 8, 2), 2, "variant prefill");
    expect(moe_gemm_variant_for(256, 4096, 14336, 8, 2), 3, "variant split");
    expect(moe_set_gemm_variant(7), -1, "bad variant");
    expect(std::strcmp(moe_status_string(3), "MOE_ERR_NO_MEMORY") == 0 ? 0 : 1, 0, "status string");
    expect(moe_version() >= 100 ? 0 : 1, 0, "version");
    // without a device the release reports the HIP error; with one it succeeds
    const int rel = moe_release_workspace();
    expect(rel == MOE_OK || rel == MOE_ERR_HIP ? 0 : 1, 0, "release");

    std::printf("abi driver: %d checks, %d failed\n", g_checks, g_fail);
    return g_fail ? 1 : 0;
}
