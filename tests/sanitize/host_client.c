/*
 * Exercises the host layer of libspeechkv.so (argument checks, overlap
 * checks, workspace sizing, split choice) under AddressSanitizer and
 * UndefinedBehaviorSanitizer.  Pointers are fake, 16-byte aligned device
 * addresses that are never dereferenced on these paths: every call here is
 * either rejected by a host check, or (with the argument "nodevice", on a
 * machine without a GPU) passes every check and fails at the device, which
 * returns SPEECHKV_ERR_HIP.  Prints "ok <count>" when every call returned
 * what it should.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "speechkv.h"

#define P(x) ((void*)(uintptr_t)(x))
#define FAKE 0x10000000ull

static int checks = 0, failures = 0;

static void expect(int got, int want, const char* what) {
  ++checks;
  if (got != want) {
    ++failures;
    printf("FAIL %s: got %d want %d\n", what, got, want);
  }
}

static speechkv_paged_kv cache(void) {
  speechkv_paged_kv c;
  c.k_pages = P(FAKE);
  c.v_pages = P(FAKE + (1ull << 24));
  c.block_table = (const int32_t*)P(FAKE + (2ull << 24));
  c.num_pages = 64;
  c.page_size = 16;
  c.max_pages_per_seq = 8;
  c.num_kv_heads = 2;
  c.head_dim = 64;
  c.dtype = SPEECHKV_DTYPE_BF16;
  return c;
}

static speechkv_spans spans(void) {
  speechkv_spans s;
  s.prefix_len = (const int32_t*)P(FAKE + (3ull << 24));
  s.speech_len = (const int32_t*)P(FAKE + (3ull << 24) + 64);
  s.suffix_len = (const int32_t*)P(FAKE + (3ull << 24) + 128);
  s.max_speech_len = 40;
  s.max_total_len = 60;
  return s;
}

static speechkv_segments segments(void) {
  speechkv_segments g;
  g.seg_start = (const int32_t*)P(FAKE + (25ull << 24));
  g.text_len = (const int32_t*)P(FAKE + (25ull << 24) + 256);
  g.speech_len = (const int32_t*)P(FAKE + (25ull << 24) + 512);
  g.num_segments = 6;
  g.max_segments = 3;
  g.max_total_len = 60;
  return g;
}

#define RAW (FAKE + (8ull << 24))
#define Q (FAKE + (9ull << 24))
#define CLEN (FAKE + (10ull << 24))
#define OUT (FAKE + (11ull << 24))
#define WS (FAKE + (14ull << 24))
#define KN (FAKE + (15ull << 24))
#define VN (FAKE + (16ull << 24))

static int pool(speechkv_paged_kv c, speechkv_spans s, uint64_t k, int32_t w, uint64_t clen) {
  return speechkv_pool_kv(P(k), P(RAW + (1 << 22)), 60 * 2 * 64, 2 * 64, 64, 2, 60, &s, w, NULL, 1,
                          0, &c, (int32_t*)P(clen), NULL);
}

static int decode(speechkv_paged_kv c, uint64_t q, uint64_t out, uint64_t kn, uint64_t vn,
                  int32_t splits, uint64_t ws, size_t ws_bytes) {
  return speechkv_decode_attn(P(q), 2, 4, &c, (const int32_t*)P(CLEN), 100, P(kn), P(vn), 0.125f,
                              splits, P(out), P(ws), ws_bytes, NULL);
}

static int prefill(speechkv_paged_kv c, speechkv_spans s, uint64_t out, uint64_t lse) {
  return speechkv_prefill_attn(P(FAKE + (12ull << 24)), 2, 4, 60, &c, &s, 4, 1, 0, 0, 0.125f, P(out),
                               (float*)P(lse), NULL);
}

int main(int argc, char** argv) {
  const int nodevice = argc > 1 && strcmp(argv[1], "nodevice") == 0;
  const speechkv_paged_kv c = cache();
  const speechkv_spans s = spans();
  speechkv_paged_kv bad = c;
  speechkv_spans sbad = s;
  const speechkv_segments g = segments();

  /* helpers */
  expect((int)speechkv_compressed_len(32, 750, 0, 4, 14, 14), 32 + 188, "compressed_len");
  expect((int)speechkv_compressed_len(-1, 3, 0, 4, 0, 0), -1, "compressed_len negative");
  {
    const int32_t t[4] = {32, 24, 16, 64}, sp[4] = {375, 250, 500, 0};
    expect((int)speechkv_compressed_len_segments(t, sp, 4, 4, 1, 0), 32 + 94 + 24 + 63 + 16 + 125 + 64,
           "compressed_len_segments");
  }
  expect(speechkv_decode_num_splits(0, 8, 10), -1, "num_splits batch 0");
  for (int b = 1; b <= 64; b *= 2)
    for (int L = 0; L <= 70000; L += 997) {
      const int n = speechkv_decode_num_splits(b, 8, L);
      ++checks;
      if (n < 1 || n > 32 || (n & (n - 1))) {
        ++failures;
        printf("FAIL num_splits(%d, 8, %d) = %d\n", b, L, n);
      }
      (void)speechkv_decode_workspace_bytes(b, 16, 8, 128, L, 0);
    }
  for (int code = 1; code >= -8; --code) (void)speechkv_status_string(code);
  (void)speechkv_version();
  expect((int)speechkv_prefill_attn_bwd_workspace_bytes(8, 16, 1596), 8 * 16 * 1596 * 4, "bwd ws");
  (void)speechkv_pool_kv_bwd_workspace_bytes(64, 782, 8, 128);
  (void)speechkv_pool_kv_bwd_workspace_bytes(2, 60, 3, 128);

  /* rejections */
  expect(pool(c, s, RAW, 0, 0), SPEECHKV_ERR_INVALID_ARG, "pool w = 0");
  expect(pool(c, s, FAKE, 4, 0), SPEECHKV_ERR_ALIAS, "pool raw in pool");
  expect(pool(c, s, RAW, 4, FAKE + 256), SPEECHKV_ERR_ALIAS, "pool lengths in pool");
  bad.head_dim = 96;
  expect(pool(bad, s, RAW, 4, 0), SPEECHKV_ERR_UNSUPPORTED, "pool head_dim");
  expect(decode(bad, Q, OUT, 0, 0, 0, 0, 0), SPEECHKV_ERR_UNSUPPORTED, "decode head_dim");
  bad = c;
  bad.v_pages = P(FAKE + 4096);
  expect(pool(bad, s, RAW, 4, 0), SPEECHKV_ERR_ALIAS, "pool pools overlap");
  expect(decode(bad, Q, OUT, KN, VN, 0, 0, 0), SPEECHKV_ERR_ALIAS, "decode pools overlap");
  sbad.max_total_len = -1;
  expect(pool(c, sbad, RAW, 4, 0), SPEECHKV_ERR_INVALID_ARG, "pool spans");
  expect(prefill(c, sbad, OUT, 0), SPEECHKV_ERR_INVALID_ARG, "prefill spans");
  expect(decode(c, Q, Q + 256, 0, 0, 0, 0, 0), SPEECHKV_ERR_ALIAS, "decode out over q");
  expect(decode(c, Q, OUT, KN, VN, 4, 0, 0), SPEECHKV_ERR_WORKSPACE, "decode no workspace");
  expect(decode(c, Q, OUT, KN, VN, 4, Q, 1 << 20), SPEECHKV_ERR_ALIAS, "decode workspace over q");
  expect(decode(c, FAKE + 2048, OUT, KN, VN, 0, 0, 0), SPEECHKV_ERR_ALIAS, "decode q in written pool");
  expect(speechkv_decode_attn_noalloc(P(Q), 8, 4, &c, (const int32_t*)P(CLEN), 100, NULL, NULL,
                                      0.125f, 4096, P(OUT), NULL),
         SPEECHKV_ERR_SCRATCH, "noalloc beyond scratch");
  expect(prefill(c, s, FAKE + 64, 0), SPEECHKV_ERR_ALIAS, "prefill out in pool");
  expect(prefill(c, s, OUT, OUT + 128), SPEECHKV_ERR_ALIAS, "prefill lse over out");
  expect(speechkv_prefill_attn_segments(P(FAKE + (12ull << 24)), 2, 4, 60, &c, &g, 4, 1, 0, 0, 0.125f,
                                        P(FAKE + (25ull << 24)), NULL, NULL),
         SPEECHKV_ERR_ALIAS, "prefill segments out over table");
  expect(speechkv_pool_kv_segments(P(RAW), P(RAW + (1 << 22)), 60 * 2 * 64, 2 * 64, 64, 2, 60, &g, 0,
                                   NULL, 1, 0, &c, NULL, NULL),
         SPEECHKV_ERR_INVALID_ARG, "pool segments w = 0");
  expect(speechkv_pool_hidden(P(FAKE + (14ull << 24)), 60 * 2048, 2048, 2, 60, 2048,
                              SPEECHKV_DTYPE_BF16, &s, 4, NULL, P(FAKE + (14ull << 24) + 4096),
                              60 * 2048, 2048, 60, NULL, NULL),
         SPEECHKV_ERR_ALIAS, "pool_hidden out over h");
  expect(speechkv_pool_prefill_attn(P(FAKE + (23ull << 24)), 2, 4, 60, P(RAW), P(RAW + (1 << 22)),
                                    60 * 2 * 64, 2 * 64, 64, 60, &s, 4, NULL, 1, 0, &c, NULL, 0,
                                    0.125f, P(RAW), NULL, NULL),
         SPEECHKV_ERR_ALIAS, "fused out over raw");
  expect(speechkv_prefill_attn_bwd(P(FAKE + (15ull << 24)), 2, 4, 60, &c, &s, 4, 1, 0, 0, 0.125f,
                                   P(FAKE + (16ull << 24)), (const float*)P(FAKE + (17ull << 24)),
                                   P(FAKE + (18ull << 24)), P(FAKE + (15ull << 24)),
                                   (float*)P(FAKE + (20ull << 24)), (float*)P(FAKE + (21ull << 24)),
                                   60, P(FAKE + (22ull << 24)), 1 << 20, NULL),
         SPEECHKV_ERR_ALIAS, "bwd dq over q");
  expect(speechkv_pool_kv_bwd(P(RAW), P(RAW + (1 << 22)), 60 * 2 * 64, 2 * 64, 64, 2, 60, 2, 64,
                              SPEECHKV_DTYPE_BF16, &s, 4, NULL, 1, 0, (const float*)P(FAKE + (23ull << 24)),
                              (const float*)P(FAKE + (24ull << 24)), 60, P(RAW), P(FAKE + (26ull << 24)),
                              NULL, NULL, 0, NULL),
         SPEECHKV_ERR_ALIAS, "pool bwd dk over raw");

  /* valid calls: every host check passes, the device is missing */
  if (nodevice) {
    const int E = SPEECHKV_ERR_HIP;
    expect(pool(c, s, RAW, 4, FAKE + (20ull << 24)), E, "valid pool");
    expect(decode(c, Q, OUT, 0, 0, 0, 0, 0), E, "valid decode");
    expect(decode(c, Q, OUT, KN, VN, 4, WS, 1 << 20), E, "valid decode, new token, splits");
    expect(speechkv_decode_attn_noalloc(P(Q), 2, 4, &c, (const int32_t*)P(CLEN), 100, P(KN), P(VN),
                                        0.125f, 4, P(OUT), NULL),
           E, "valid noalloc");
    expect(prefill(c, s, OUT, FAKE + (20ull << 24)), E, "valid prefill");
    expect(speechkv_prefill_attn_segments(P(FAKE + (12ull << 24)), 2, 4, 60, &c, &g, 4, 1, 0, 0,
                                          0.125f, P(OUT), NULL, NULL),
           E, "valid prefill segments");
    expect(speechkv_pool_kv_segments(P(RAW), P(RAW + (1 << 22)), 60 * 2 * 64, 2 * 64, 64, 2, 60, &g,
                                     4, NULL, 1, 0, &c, NULL, NULL),
           E, "valid pool segments");
    expect(speechkv_pool_prefill_attn(P(FAKE + (23ull << 24)), 2, 4, 60, P(RAW), P(RAW + (1 << 22)),
                                      60 * 2 * 64, 2 * 64, 64, 60, &s, 4, NULL, 1, 0, &c, NULL, 0,
                                      0.125f, P(FAKE + (24ull << 24)), NULL, NULL),
           E, "valid fused");
    expect(speechkv_prefill_attn_bwd(P(FAKE + (15ull << 24)), 2, 4, 60, &c, &s, 4, 1, 0, 0, 0.125f,
                                     P(FAKE + (16ull << 24)), (const float*)P(FAKE + (17ull << 24)),
                                     P(FAKE + (18ull << 24)), P(FAKE + (19ull << 24)),
                                     (float*)P(FAKE + (20ull << 24)), (float*)P(FAKE + (21ull << 24)),
                                     60, P(FAKE + (22ull << 24)), 1 << 20, NULL),
           E, "valid bwd");
    expect(speechkv_pool_kv_bwd(P(RAW), P(RAW + (1 << 22)), 60 * 2 * 64, 2 * 64, 64, 2, 60, 2, 64,
                                SPEECHKV_DTYPE_BF16, &s, 4, NULL, 1, 0,
                                (const float*)P(FAKE + (23ull << 24)),
                                (const float*)P(FAKE + (24ull << 24)), 60, P(FAKE + (25ull << 24)),
                                P(FAKE + (26ull << 24)), NULL, NULL, 0, NULL),
           E, "valid pool bwd");
    expect(speechkv_pool_hidden(P(FAKE + (14ull << 24)), 60 * 2048, 2048, 2, 60, 2048,
                                SPEECHKV_DTYPE_BF16, &s, 4, NULL, P(FAKE + (30ull << 24)), 60 * 2048,
                                2048, 60, NULL, NULL),
           E, "valid pool_hidden");
  }
  printf("%s %d\n", failures ? "failed" : "ok", checks);
  return failures ? 1 : 0;
}
