// Host-side argument checks of every C-ABI entry point, run without a GPU in a build of the
// library whose host code has AddressSanitizer and UBSan (tests/test_abi_sanitized.py). Each
// call below must return the status it names before anything reaches the device; calls that
// pass every check return PG_EHIP here (no device). Prints one line per mismatch and exits 1.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include "pg_attn.h"

static int g_bad = 0;
static void expect(const char* what, int got, int want) {
  if (got != want) {
    printf("MISMATCH %s: got %d want %d (%s)\n", what, got, want, pg_last_error());
    ++g_bad;
  }
}

int main() {
  // dummy non-null pointers: every call below fails before dereferencing them
  const int32_t* ip = reinterpret_cast<const int32_t*>(uintptr_t(64));
  void* p = reinterpret_cast<void*>(uintptr_t(64));
  float* fp = reinterpret_cast<float*>(uintptr_t(64));
  const size_t big = size_t(1) << 40;
  const float nan = std::numeric_limits<float>::quiet_NaN(), inf = std::numeric_limits<float>::infinity();

  struct F {
    int dt, ng, ns, tp, ts, hq, hkv, d;
    float sc;
    bool null_grp, null_t;
    size_t ws;
    int want;
    const char* what;
  };
  const F cases[] = {
      {7, 1, 2, 8, 6, 4, 2, 128, .1f, false, false, big, PG_EUNSUPPORTED, "dtype"},
      {0, -1, 2, 8, 6, 4, 2, 128, .1f, false, false, big, PG_EINVAL, "negative groups"},
      {0, 1, 2, -8, 6, 4, 2, 128, .1f, false, false, big, PG_EINVAL, "negative prefix"},
      {0, 0, 0, 8, 0, 4, 2, 128, .1f, false, false, big, PG_EINVAL, "prefix rows without groups"},
      {0, 1, 0, 8, 6, 4, 2, 128, .1f, false, false, big, PG_EINVAL, "response rows without members"},
      {0, 1, 2, 8, 6, 5, 2, 128, .1f, false, false, big, PG_EINVAL, "h_q % h_kv"},
      {0, 1, 2, 8, 6, 0, 0, 128, .1f, false, false, big, PG_EINVAL, "zero heads"},
      {0, 1, 2, 8, 6, 4, 2, 96, .1f, false, false, big, PG_EUNSUPPORTED, "head_dim"},
      {0, 1, 2, 8, 6, 1024, 2, 128, .1f, false, false, big, PG_EUNSUPPORTED, "h_q * head_dim"},
      {0, 1, 2, 8, 6, 4, 2, 128, nan, false, false, big, PG_EINVAL, "NaN scale"},
      {0, 1, 2, 8, 6, 4, 2, 128, inf, false, false, big, PG_EINVAL, "inf scale"},
      {0, 1, 2, 8, 6, 4, 2, 128, 0.f, false, false, big, PG_EINVAL, "zero scale"},
      {0, 1, 2, 8, 6, 4, 2, 128, -1.f, false, false, big, PG_EINVAL, "negative scale"},
      {0, 1, 2, 0x7fffffff, 6, 4, 2, 128, .1f, false, false, big, PG_EUNSUPPORTED, "rows * h_q > 2^31"},
      {0, 1, 2, 8, 6, 4, 2, 128, .1f, true, false, big, PG_EINVAL, "null grouping arrays"},
      {0, 1, 2, 8, 6, 4, 2, 128, .1f, false, true, big, PG_EINVAL, "null tensors"},
      {0, 1, 2, 8, 6, 4, 2, 128, .1f, false, false, 16, PG_EWORKSPACE, "small workspace"},
      {0, 1, 2, 8, 6, 4, 2, 128, .1f, false, false, 0, PG_EWORKSPACE, "no workspace"},
      {1, 1, 2, 8, 6, 4, 2, 64, .1f, false, false, big, PG_EHIP, "valid (no device here)"},
  };
  for (const F& c : cases) {
    const int32_t* g = c.null_grp ? nullptr : ip;
    void* t = c.null_t ? nullptr : p;
    float* tl = c.null_t ? nullptr : fp;
    void* ws = c.ws ? p : nullptr;
    char name[160];
    snprintf(name, sizeof name, "fwd %s", c.what);
    expect(name, pg_attn_fwd(c.dt, c.ng, c.ns, c.tp, c.ts, g, g, g, c.hq, c.hkv, c.d, c.sc, t, t, t, t, t, t, t, t,
                             tl, tl, ws, c.ws, nullptr), c.want);
    snprintf(name, sizeof name, "bwd %s", c.what);
    expect(name, pg_attn_bwd(c.dt, c.ng, c.ns, c.tp, c.ts, g, g, g, c.hq, c.hkv, c.d, c.sc, t, t, t, t, t, t, t, t,
                             tl, tl, t, t, t, t, t, t, t, t, ws, c.ws, nullptr), c.want);
    snprintf(name, sizeof name, "fwd_xours %s", c.what);
    expect(name, pg_attn_fwd_xours(c.dt, c.ng, c.ns, c.tp, c.ts, g, g, g, c.hq, c.hkv, c.d, c.sc, t, t, t, t, tl, ws,
                                   c.ws, nullptr), c.want);
    snprintf(name, sizeof name, "bwd_xours %s", c.what);
    expect(name, pg_attn_bwd_xours(c.dt, c.ng, c.ns, c.tp, c.ts, g, g, g, c.hq, c.hkv, c.d, c.sc, t, t, t, t, tl, t, t,
                                   t, t, ws, c.ws, nullptr), c.want);
  }
  // final-token forward: its own limit on the heads per kv head, and its workspace
  expect("last ratio", pg_attn_fwd_last(0, 1, 2, 8, 6, ip, ip, ip, 256, 1, 128, .1f, p, p, p, p, p, p, p, fp, p, big,
                                        nullptr), PG_EUNSUPPORTED);
  expect("last null outputs", pg_attn_fwd_last(0, 1, 2, 8, 6, ip, ip, ip, 4, 2, 128, .1f, p, p, p, p, p, p, nullptr,
                                               nullptr, p, big, nullptr), PG_EINVAL);
  expect("last small workspace", pg_attn_fwd_last(0, 1, 2, 8, 6, ip, ip, ip, 4, 2, 128, .1f, p, p, p, p, p, p, p, fp,
                                                  p, 8, nullptr), PG_EWORKSPACE);
  // rotary embedding
  expect("rope rotary_dim", pg_rope(0, 1, 2, 8, 6, ip, ip, ip, 4, 2, 128, 8, 1e4, 0, p, p, p, p, p, p, p, p, p, big,
                                    nullptr), PG_EUNSUPPORTED);
  expect("rope base", pg_rope(0, 1, 2, 8, 6, ip, ip, ip, 4, 2, 128, 128, -1.0, 0, p, p, p, p, p, p, p, p, p, big,
                              nullptr), PG_EINVAL);
  expect("rope flags", pg_rope(0, 1, 2, 8, 6, ip, ip, ip, 4, 2, 128, 128, 1e4, 8, p, p, p, p, p, p, p, p, p, big,
                               nullptr), PG_EINVAL);
  void* odd = reinterpret_cast<void*>(uintptr_t(66));
  expect("rope alignment", pg_rope(0, 1, 2, 8, 6, ip, ip, ip, 4, 2, 128, 128, 1e4, 0, odd, p, p, p, p, p, p, p, p, big,
                                   nullptr), PG_EINVAL);
  expect("rope heads", pg_rope(0, 1, 2, 8, 6, ip, ip, ip, 0, 0, 128, 128, 1e4, 0, p, p, p, p, p, p, p, p, p, big,
                               nullptr), PG_EINVAL);
  expect("positions null", pg_grouped_positions(1, 2, 8, 6, ip, ip, ip, nullptr, nullptr, p, big, nullptr), PG_EINVAL);
  expect("positions workspace", pg_grouped_positions(1, 2, 8, 6, ip, ip, ip, (int32_t*)p, (int32_t*)p, p, 1, nullptr),
         PG_EWORKSPACE);
  // size queries: negative sizes give 0, the largest legal ones a finite size
  if (pg_attn_fwd_workspace_size(-1, 0, 0, 0, 1, 1, 64) != 0) { printf("MISMATCH fwd size of negative\n"); ++g_bad; }
  if (pg_attn_bwd_workspace_size(1, 1, 0x7fffffff, 0x7fffffff, 1, 1, 128) == 0) {
    printf("MISMATCH bwd size of the largest sizes\n");
    ++g_bad;
  }
  if (pg_attn_fwd_last_workspace_size(0x7fffffff, 0x7fffffff, 0, 0, 1, 1, 128) == 0) {
    printf("MISMATCH last size of the largest sizes\n");
    ++g_bad;
  }
  if (pg_rope_workspace_size(0x7fffffff) == 0) { printf("MISMATCH rope size\n"); ++g_bad; }
  expect("plan status small workspace", pg_plan_status(p, 16, nullptr), PG_EWORKSPACE);
  // status strings and timing queries
  for (int s = -1; s <= 5; ++s)
    if (!pg_status_string(s) || !*pg_status_string(s)) { printf("MISMATCH status string %d\n", s); ++g_bad; }
  expect("timing null", pg_timing_get(1, nullptr, nullptr), PG_EINVAL);
  int n = -1;
  double ms = -1;
  expect("timing start", pg_timing_start(), PG_OK);
  expect("timing get", pg_timing_get(1, &n, &ms), PG_OK);
  expect("timing stop", pg_timing_stop(), PG_OK);
  if (n != 0) { printf("MISMATCH timing launches %d\n", n); ++g_bad; }
  printf("%s (%d mismatches)\n", g_bad ? "FAIL" : "OK", g_bad);
  return g_bad ? 1 : 0;
}
