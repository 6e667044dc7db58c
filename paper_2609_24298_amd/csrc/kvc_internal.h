// Internal declarations shared by the host (kvc_host.cpp) and device (kvc_kernels.hip)
// halves of libkvc. Not part of the public ABI.
#pragma once

#include <cstdint>

#include "kvc.h"

namespace kvc {

// Records a thread-local error message and returns `code`.
int set_error(int code, const char* fmt, ...);
// Clears the thread-local error message.
void clear_error();

// Host-side checks of a stream descriptor (pointers, per-unit r/b/offset/step
// ranges, arena bounds for `capacity` tokens). Returns KVC_OK or an error.
int validate_desc(const kvc_stream_desc* s, const char* name);

// Bytes of a stream holding n_tok tokens: whole 64-token tiles of 8*r*b bytes.
inline int64_t stream_bytes(int64_t n_tok, int r, int b) {
    return ((n_tok + KVC_TILE_TOKENS - 1) / KVC_TILE_TOKENS) * 8LL * r * b;
}

}  // namespace kvc
