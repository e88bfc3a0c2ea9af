// Library-internal helpers shared by the C-ABI translation units (not
// exported: the library is built with hidden visibility).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ws.h"

namespace ws_internal {

// Records the message for ws_last_error() and returns st.
ws_status fail(ws_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
ws_status hip_fail(hipError_t e, const char* what);

int32_t cache_heads(const ws_cache* c);
int32_t cache_max_q(const ws_cache* c);

// Checks, without changing anything, that ws_step_append could take a
// segment of n_tokens for (unit, kind): a fresh segment needs free pages
// (pages_needed accumulates them), a rewrite needs an uncommitted segment of
// the same length.
ws_status precheck_append(const ws_cache* c, int32_t unit, ws_kind kind, int32_t n_tokens,
                          int32_t* pages_needed);
int32_t free_pages(const ws_cache* c);

// Launch timing ring (ws_cache_timing_*): a slot for one call of `path`,
// its first event recorded (unless `stamped`: the call's kernel launch takes
// events 0 and 1 as its dispatch's start and end); timing_mark records event
// k (0, 1, 2) of the slot.
ws_status timing_begin_path(ws_cache* c, int32_t path, int32_t splits, hipStream_t stream, int* slot,
                            bool stamped = false);
ws_status timing_mark(ws_cache* c, int slot, int k, hipStream_t stream);

}  // namespace ws_internal
