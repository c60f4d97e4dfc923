// Host-side argument checks of libbs_attn's C ABI under the address and undefined-behaviour
// sanitizers: every call below fails validation before the library touches a device (the
// pointers are placeholders that are never dereferenced), so it runs without a GPU.  Built by
// tests/test_capi_sanitized.py with capi.hip instrumented on the host side only.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../include/bs_attn.h"

#define CHECK(cond)                                                                   \
  do {                                                                                \
    if (!(cond)) {                                                                    \
      std::fprintf(stderr, "check failed: %s (last error: %s)\n", #cond, bs_last_error()); \
      std::exit(1);                                                                   \
    }                                                                                 \
  } while (0)

static void* const FAKE = reinterpret_cast<void*>(4096);

static bs_dims dims(int64_t tq = 128, int32_t hq = 4, int32_t hkv = 2, int32_t d = 128,
                    int dtype = BS_BF16) {
  bs_dims x;
  std::memset(&x, 0, sizeof(x));
  x.total_q = tq;
  x.total_k = tq;
  x.hq = hq;
  x.hkv = hkv;
  x.head_dim = d;
  x.dtype = (bs_dtype)dtype;
  return x;
}

static int fwd(const bs_dims& d, size_t ws_bytes = (size_t)1 << 30, float scale = 0.1f,
               const void* q = FAKE, const int32_t* cu = (const int32_t*)FAKE) {
  return bs_attn_varlen_fwd(&d, q, FAKE, FAKE, cu, cu, 1, 128, 1, scale, FAKE, (float*)FAKE, FAKE,
                            ws_bytes, nullptr);
}

int main() {
  CHECK(fwd(dims(128, 4, 2, 96)) == BS_ERR_UNSUPPORTED);
  CHECK(std::strstr(bs_last_error(), "head_dim") != nullptr);
  CHECK(fwd(dims(128, 4, 2, 128, 7)) == BS_ERR_UNSUPPORTED);
  CHECK(fwd(dims(128, 6, 4)) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(128, 4, 0)) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(128, 8192, 8)) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(-1)) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(), (size_t)1 << 30, 0.1f, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(), (size_t)1 << 30, 0.1f, (const char*)FAKE + 2) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(), (size_t)1 << 30, NAN) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(), (size_t)1 << 30, -1.0f) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(), (size_t)1 << 30, 0.1f, FAKE, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(fwd(dims(), 16) == BS_ERR_WORKSPACE);
  CHECK(std::strstr(bs_last_error(), "smaller") != nullptr);

  const bs_dims d = dims();
  CHECK(bs_lse_merge(&d, FAKE, (const float*)FAKE, 0, FAKE, (float*)FAKE, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_read_device_status(nullptr, nullptr) == BS_ERR_WORKSPACE);
  CHECK(bs_copy_async(nullptr, FAKE, 64, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_copy_async(FAKE, (char*)FAKE + 32, 64, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_copy_async(nullptr, nullptr, 0, nullptr) == BS_OK);

  // fused cross-entropy
  CHECK(bs_softmax_xent(4, 1000, 5, FAKE, (const int64_t*)FAKE, -100, 1.0f, (float*)FAKE, nullptr,
                        nullptr, nullptr) == BS_ERR_UNSUPPORTED);
  CHECK(bs_softmax_xent(-1, 1000, BS_BF16, FAKE, (const int64_t*)FAKE, -100, 1.0f, (float*)FAKE,
                        nullptr, nullptr, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_softmax_xent(4, 0, BS_BF16, FAKE, (const int64_t*)FAKE, -100, 1.0f, (float*)FAKE,
                        nullptr, nullptr, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_softmax_xent(4, 1000, BS_BF16, (const char*)FAKE + 1, (const int64_t*)FAKE, -100, 1.0f,
                        (float*)FAKE, nullptr, nullptr, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_softmax_xent(4, 1000, BS_BF16, FAKE, (const int64_t*)FAKE, -100, INFINITY,
                        (float*)FAKE, nullptr, nullptr, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_softmax_xent(4, 1000, BS_BF16, FAKE, (const int64_t*)FAKE, -100, 1.0f, (float*)FAKE,
                        nullptr, (char*)FAKE + 64, nullptr) == BS_ERR_INVALID_ARG);
  CHECK(bs_softmax_xent(0, 1000, BS_BF16, nullptr, nullptr, -100, 1.0f, nullptr, nullptr, nullptr,
                        nullptr) == BS_OK);

  // running merge: both running buffers, no overlap with the final output
  const int64_t qn = 128 * 4 * 128;
  auto chunk = [&](void* o_run, void* lse_run, void* out, size_t ws) {
    return bs_attn_chunk_fwd_merge(&d, FAKE, FAKE, FAKE, 0, 0, 1, 0.1f, (float*)o_run,
                                   (float*)lse_run, 1, out, FAKE, ws, nullptr);
  };
  char* base = reinterpret_cast<char*>(1 << 20);
  CHECK(chunk(nullptr, FAKE, nullptr, (size_t)1 << 30) == BS_ERR_INVALID_ARG);
  CHECK(chunk(FAKE, nullptr, nullptr, (size_t)1 << 30) == BS_ERR_INVALID_ARG);
  CHECK(chunk((char*)FAKE + 8, FAKE, nullptr, (size_t)1 << 30) == BS_ERR_INVALID_ARG);
  CHECK(chunk(base, FAKE, base + qn * 4 - 16, (size_t)1 << 30) == BS_ERR_INVALID_ARG);
  CHECK(chunk(base, FAKE, base + qn * 4, 16) == BS_ERR_WORKSPACE);

  // workspace sizes
  const bs_dims big = dims(4096);
  const size_t s_small = bs_attn_workspace_size(BS_OP_VARLEN_FWD, &d, 1, 128);
  const size_t s_big = bs_attn_workspace_size(BS_OP_VARLEN_FWD, &big, 1, 4096);
  const size_t s_bwd = bs_attn_workspace_size(BS_OP_VARLEN_BWD, &big, 1, 4096);
  CHECK(0 < s_small && s_small < s_big && s_big < s_bwd);
  CHECK(bs_attn_workspace_size(9, &d, 1, 1) == 0);

  // the allocation-free forward: sizes beyond its scratch array
  const bs_dims huge = dims((int64_t)1 << 28);
  CHECK(bs_attn_varlen_fwd_noalloc(&huge, FAKE, FAKE, FAKE, (const int32_t*)FAKE,
                                   (const int32_t*)FAKE, 1, 1 << 28, 1, 0.1f, FAKE, (float*)FAKE,
                                   nullptr) == BS_ERR_WORKSPACE);
  CHECK(std::strstr(bs_last_error(), "allocation-free") != nullptr);
  CHECK(bs_attn_varlen_fwd_noalloc(&d, FAKE, FAKE, FAKE, nullptr, nullptr, 1, 128, 1, 0.1f, FAKE,
                                   (float*)FAKE, nullptr) == BS_ERR_INVALID_ARG);
  // a long error message is truncated, not overflowed
  for (int i = 0; i < 1000; ++i) CHECK(fwd(dims(128, 4, 2, 96)) == BS_ERR_UNSUPPORTED);
  std::printf("ok\n");
  return 0;
}
