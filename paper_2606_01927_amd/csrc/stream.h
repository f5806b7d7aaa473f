// stream.h -- internal interface between the C ABI (albireo.hip) and the streaming sampling kernel
// (stream.hip).  Not part of the public header: the public sampling entry points route here.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "albireo.h"

namespace albireo_stream {

// Everything one sampling launch needs (device pointers unless noted).
struct Request {
  const void* logits;
  albireo_dtype_t dtype;
  int64_t B, V, ld;
  const albireo_params_t* params;  // [host] or NULL
  const float* uniforms;           // NULL when step is given
  const albireo_step_t* step;      // [host] or NULL
  const albireo_shards_t* shards;  // [host] or NULL (row-major)
  int32_t* out_ids;
  float* out_logprobs;
  int32_t n_top;
  int32_t* out_top_ids;
  float* out_top_logprobs;
  uint32_t* out_flags;
  unsigned char* ws;  // the caller's workspace (256-byte aligned), workspace_bytes(B, V, dtype) long
  hipStream_t stream;
};

// Whether the kernel handles rows of this shape (V, dtype, batch size).
bool supported(int64_t B, int64_t V, albireo_dtype_t dtype);

// Workspace bytes the kernel needs for B rows (0 when not supported).  The bytes must be zero before a
// call, and the kernel leaves every byte it wrote zero again (the workspace contract of the public
// header), so one workspace serves every entry point and shape in turn.
size_t workspace_bytes(int64_t B, int64_t V, albireo_dtype_t dtype);

// Enqueue one launch.  The caller has validated every host-checkable argument.
albireo_status_t launch(const Request& r);

}  // namespace albireo_stream
