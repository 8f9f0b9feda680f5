/*
 * Runs every entry point of the fp64 oracle (oracle/moe_oracle.c) once on
 * small deterministic inputs, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer.  Inputs and outputs are written to the file
 * named by argv[1] as a sequence of records
 *   u32 name length, name bytes, u32 type code, u64 byte count, bytes
 * (type codes: 1 u16, 2 u8, 3 f32, 4 f64, 5 i32), so that the test can run
 * the same calls through the normal build and compare the bits.
 *
 * Inputs come from a 64-bit linear congruential generator (Knuth's MMIX
 * constants); bf16 values are the top halves of floats in [-1, 1), E4M3
 * bytes avoid the two NaN codes.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_threads(int n);
int oracle_router_logits(const uint16_t* x, const uint16_t* wr, const float* bias, int64_t T,
                         int64_t d, int64_t E, double* logits);
int oracle_topk_gate(const double* logits, int64_t T, int E, int k, int32_t* ids, double* gates);
int oracle_gates_for_ids(const double* logits, const int32_t* ids, int64_t T, int E, int k,
                         double* gates);
int oracle_dispatch(const int32_t* ids, int64_t T, int E, int k, int32_t* counts,
                    int32_t* offsets, int32_t* perm);
int oracle_moe_apply(const uint16_t* x, const uint16_t* w1, const uint16_t* w3,
                     const uint16_t* w2, const int32_t* ids, const double* gates, int64_t T,
                     int64_t d, int64_t ffn, int E, int k, double* out, double* h_slots,
                     double* y_slots);
int oracle_moe_layer(const uint16_t* x, const uint16_t* wr, const float* bias, const uint16_t* w1,
                     const uint16_t* w3, const uint16_t* w2, int64_t T, int64_t d, int64_t ffn,
                     int E, int k, double* out, double* logits, int32_t* ids, double* gates);
int oracle_fp8_e4m3(const uint8_t* q, int64_t n, double* out);
int oracle_moe_apply_fp8(const uint16_t* x, const uint8_t* w1q, const float* w1s,
                         const uint8_t* w3q, const float* w3s, const uint8_t* w2q,
                         const float* w2s, const int32_t* ids, const double* gates, int64_t T,
                         int64_t d, int64_t ffn, int E, int k, double* out, double* h_slots,
                         double* y_slots);
int oracle_moe_layer_fp8(const uint16_t* x, const uint16_t* wr, const float* bias,
                         const uint8_t* w1q, const float* w1s, const uint8_t* w3q,
                         const float* w3s, const uint8_t* w2q, const float* w2s, int64_t T,
                         int64_t d, int64_t ffn, int E, int k, double* out, double* logits,
                         int32_t* ids, double* gates);
int oracle_rmsnorm(const float* h, const uint16_t* gamma, int64_t T, int64_t d, double eps,
                   double* a);
int oracle_round_bf16(const double* x, int64_t n, uint16_t* out);
int oracle_rope(double* x, int64_t T, int H, int hd, const int32_t* pos, double base);
int oracle_attention_decode(const double* q, const uint16_t* kc, const uint16_t* vc,
                            const int32_t* page_table, int64_t maxp, int64_t npages,
                            const int32_t* ctx, int64_t T, int Hq, int Hkv, int hd, int page,
                            double scale, double* out);

static uint64_t g_state = 2408;
static uint64_t next_u64(void)
{
    g_state = g_state * 6364136223846793005ULL + 1442695040888963407ULL;
    return g_state;
}
static float uniform(void) { return (float)((next_u64() >> 40) * (1.0 / 16777216.0)) * 2.0f - 1.0f; }
static uint16_t bf16_of(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

static FILE* g_out;
static void put(const char* name, int type, const void* p, size_t bytes)
{
    uint32_t n = (uint32_t)strlen(name), t = (uint32_t)type;
    uint64_t b = bytes;
    if (fwrite(&n, 4, 1, g_out) != 1 || fwrite(name, 1, n, g_out) != n ||
        fwrite(&t, 4, 1, g_out) != 1 || fwrite(&b, 8, 1, g_out) != 1 ||
        (bytes && fwrite(p, 1, bytes, g_out) != bytes)) {
        fprintf(stderr, "write failed\n");
        exit(3);
    }
}
/* every buffer of the driver, freed before exit so that LeakSanitizer
   reports only what the oracle itself leaks */
static void* g_bufs[128];
static int g_nbufs;
static void* take(size_t bytes)
{
    void* p = calloc(bytes ? bytes : 1, 1);
    if (!p || g_nbufs == 128) exit(4);
    g_bufs[g_nbufs++] = p;
    return p;
}
static uint16_t* bf16_array(size_t n, float scale)
{
    uint16_t* a = take(n * 2);
    for (size_t i = 0; i < n; ++i) a[i] = bf16_of(uniform() * scale);
    return a;
}
static uint8_t* e4m3_array(size_t n)
{
    uint8_t* a = take(n);
    for (size_t i = 0; i < n; ++i) {
        uint8_t b = (uint8_t)(next_u64() >> 56);
        if ((b & 0x7F) == 0x7F) b ^= 1; /* not a NaN code */
        a[i] = b;
    }
    return a;
}
static float* f32_array(size_t n, float lo, float hi)
{
    float* a = take(n * 4);
    for (size_t i = 0; i < n; ++i) a[i] = lo + (hi - lo) * 0.5f * (uniform() + 1.0f);
    return a;
}

#define CHECK(call)                                                            \
    do {                                                                       \
        int rc_ = (call);                                                      \
        if (rc_ != 0) {                                                        \
            fprintf(stderr, "%s returned %d\n", #call, rc_);                   \
            return 2;                                                          \
        }                                                                      \
    } while (0)

int main(int argc, char** argv)
{
    if (argc < 2) return 1;
    g_out = fopen(argv[1], "wb");
    if (!g_out) return 1;
    oracle_threads(2);
    const int64_t T = 13, d = 128, ffn = 192;
    const int E = 8, k = 2;
    uint16_t* x = bf16_array(T * d, 2.0f);
    uint16_t* wr = bf16_array(E * d, 0.2f);
    uint16_t* w1 = bf16_array(E * ffn * d, 0.15f);
    uint16_t* w3 = bf16_array(E * ffn * d, 0.15f);
    uint16_t* w2 = bf16_array(E * d * ffn, 0.12f);
    float* bias = f32_array(E, -0.5f, 0.5f);
    put("x", 1, x, T * d * 2);
    put("wr", 1, wr, E * d * 2);
    put("w1", 1, w1, E * ffn * d * 2);
    put("w3", 1, w3, E * ffn * d * 2);
    put("w2", 1, w2, E * d * ffn * 2);
    put("bias", 3, bias, E * 4);

    double* logits = take(T * E * 8);
    CHECK(oracle_router_logits(x, wr, bias, T, d, E, logits));
    put("logits", 4, logits, T * E * 8);
    int32_t* ids = take(T * k * 4);
    double* gates = take(T * k * 8);
    CHECK(oracle_topk_gate(logits, T, E, k, ids, gates));
    put("ids", 5, ids, T * k * 4);
    put("gates", 4, gates, T * k * 8);
    /* gates of a different valid selection: the experts ranked 3rd and 1st */
    int32_t* ids2 = take(T * k * 4);
    for (int64_t t = 0; t < T; ++t) {
        ids2[t * k] = (ids[t * k] + 3) % E;
        ids2[t * k + 1] = ids[t * k];
    }
    double* gates2 = take(T * k * 8);
    CHECK(oracle_gates_for_ids(logits, ids2, T, E, k, gates2));
    put("ids2", 5, ids2, T * k * 4);
    put("gates2", 4, gates2, T * k * 8);
    int32_t* counts = take(E * 4);
    int32_t* offsets = take((E + 1) * 4);
    int32_t* perm = take(T * k * 4);
    CHECK(oracle_dispatch(ids, T, E, k, counts, offsets, perm));
    put("counts", 5, counts, E * 4);
    put("offsets", 5, offsets, (E + 1) * 4);
    put("perm", 5, perm, T * k * 4);

    double* out = take(T * d * 8);
    double* hs = take(T * k * ffn * 8);
    double* ys = take(T * k * d * 8);
    CHECK(oracle_moe_apply(x, w1, w3, w2, ids, gates, T, d, ffn, E, k, out, hs, ys));
    put("apply_out", 4, out, T * d * 8);
    put("apply_h", 4, hs, T * k * ffn * 8);
    put("apply_y", 4, ys, T * k * d * 8);
    double* lout = take(T * d * 8);
    double* llog = take(T * E * 8);
    int32_t* lids = take(T * k * 4);
    double* lg = take(T * k * 8);
    CHECK(oracle_moe_layer(x, wr, bias, w1, w3, w2, T, d, ffn, E, k, lout, llog, lids, lg));
    put("layer_out", 4, lout, T * d * 8);

    uint8_t* q1 = e4m3_array(E * ffn * d);
    uint8_t* q3 = e4m3_array(E * ffn * d);
    uint8_t* q2 = e4m3_array(E * d * ffn);
    float* s1 = f32_array(E * ffn, 0.01f, 0.03f);
    float* s3 = f32_array(E * ffn, 0.01f, 0.03f);
    float* s2 = f32_array(E * d, 0.01f, 0.03f);
    put("q1", 2, q1, E * ffn * d);
    put("q3", 2, q3, E * ffn * d);
    put("q2", 2, q2, E * d * ffn);
    put("s1", 3, s1, E * ffn * 4);
    put("s3", 3, s3, E * ffn * 4);
    put("s2", 3, s2, E * d * 4);
    uint8_t codes[256];
    for (int i = 0; i < 256; ++i) codes[i] = (uint8_t)i;
    double* widened = take(256 * 8);
    CHECK(oracle_fp8_e4m3(codes, 256, widened));
    put("e4m3_all", 4, widened, 256 * 8);
    CHECK(oracle_moe_apply_fp8(x, q1, s1, q3, s3, q2, s2, ids, gates, T, d, ffn, E, k, out, hs, ys));
    put("apply8_out", 4, out, T * d * 8);
    put("apply8_h", 4, hs, T * k * ffn * 8);
    CHECK(oracle_moe_layer_fp8(x, wr, NULL, q1, s1, q3, s3, q2, s2, T, d, ffn, E, k, lout, llog,
                               lids, lg));
    put("layer8_out", 4, lout, T * d * 8);

    float* hres = f32_array(T * d, -3.0f, 3.0f);
    uint16_t* gamma = bf16_array(d, 1.0f);
    double* a = take(T * d * 8);
    put("hres", 3, hres, T * d * 4);
    put("gamma", 1, gamma, d * 2);
    CHECK(oracle_rmsnorm(hres, gamma, T, d, 1e-5, a));
    put("rms", 4, a, T * d * 8);
    uint16_t* ab = take(T * d * 2);
    CHECK(oracle_round_bf16(a, T * d, ab));
    put("rms_bf16", 1, ab, T * d * 2);

    /* decode attention over a paged cache: 3 requests, 2 KV heads of 2 query
       heads each, head size 16, pages of 8 positions */
    const int Tq = 3, Hq = 4, Hkv = 2, hd = 16, page = 8, maxp = 4, npages = 10;
    double* q = take((size_t)Tq * Hq * hd * 8);
    for (int i = 0; i < Tq * Hq * hd; ++i) q[i] = uniform();
    put("q_in", 4, q, (size_t)Tq * Hq * hd * 8);
    int32_t pos[3] = {5, 17, 30};
    put("pos", 5, pos, sizeof pos);
    CHECK(oracle_rope(q, Tq, Hq, hd, pos, 10000.0));
    put("q_rope", 4, q, (size_t)Tq * Hq * hd * 8);
    uint16_t* kc = bf16_array((size_t)npages * Hkv * page * hd, 1.0f);
    uint16_t* vc = bf16_array((size_t)npages * Hkv * page * hd, 1.0f);
    int32_t pt[3 * 4] = {9, 0, 0, 0, 1, 3, 7, 0, 2, 4, 5, 6};
    int32_t ctx[3] = {6, 18, 31};
    put("kc", 1, kc, (size_t)npages * Hkv * page * hd * 2);
    put("vc", 1, vc, (size_t)npages * Hkv * page * hd * 2);
    put("pt", 5, pt, sizeof pt);
    put("ctx", 5, ctx, sizeof ctx);
    double* ao = take((size_t)Tq * Hq * hd * 8);
    CHECK(oracle_attention_decode(q, kc, vc, pt, maxp, npages, ctx, Tq, Hq, Hkv, hd, page, 0.25, ao));
    put("attn", 4, ao, (size_t)Tq * Hq * hd * 8);
    fclose(g_out);
    for (int i = 0; i < g_nbufs; ++i) free(g_bufs[i]);
    printf("oracle driver: all entry points ran\n");
    return 0;
}
