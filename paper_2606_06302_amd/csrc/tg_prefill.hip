// Ragged chunked-prefill attention for gfx950 (bf16 MFMA).
#include <hip/hip_runtime.h>

#include "tg_internal.h"

extern "C" {

size_t tg_prefill_workspace_bytes(const tg_prefill_args* args) {
  (void)args;
  return 0;
}

int32_t tg_prefill(const tg_prefill_args* a, void* hip_stream) {
  (void)a;
  (void)hip_stream;
  return tg::fail(TG_ERR_UNSUPPORTED, "prefill kernel not built yet");
}

}  // extern "C"
