// ts_internal.h -- host-side helpers shared by the library's translation
// units (error reporting, device check).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ts_attn.h"

namespace tsattn {

struct AttnParams;
typedef void (*kernel_fn)(AttnParams);

// Records a formatted message as the thread's last error and returns status.
int fail(int status, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int hip_fail(hipError_t e, const char *what);
void clear_error();
// TS_OK if the current device is a gfx950, else TS_ERR_UNSUPPORTED / TS_ERR_HIP.
int check_device();
// TS_OK if every field of the shape is inside the supported set (the checks
// of ts_decode_attn), else TS_ERR_NULL / TS_ERR_SHAPE with a message.
int check_shape(const ts_attn_shape *s);
// The body of ts_decode_attn / ts_decode_attn_events: validates, plans and
// enqueues the call on `stream` with the given workspace (allocates nothing).
int launch_attn(const ts_attn_shape *s, const void *q, const void *k_pages, const void *v_pages,
                const int32_t *page_table, const int32_t *ctx_lens, const int32_t *q_lens, void *out,
                float scale, void *workspace, size_t workspace_bytes, void *stream, void *ev_begin,
                void *ev_end);

}  // namespace tsattn
