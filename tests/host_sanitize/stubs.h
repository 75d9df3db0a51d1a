// Record of the stubbed launches (host sanitizer build of the host layer).
#pragma once
#include <stddef.h>

#include <hip/hip_runtime_api.h>

struct StubLog {
  int attn_bf16 = 0, attn_f32 = 0, merge = 0, accept = 0, sample = 0, tree_calls = 0, commit = 0;
  bool tree = false;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  const void* ws = nullptr;  // the workspace the next call receives
  size_t ws_bytes = 0;
};
extern StubLog g_stub;
