// Status and error text shared by the host translation units: every public
// entry point returns an ma_status_t and leaves a message for
// mesh_attn_last_error() on the calling thread.
#pragma once

#include "mesh_attn.h"

namespace mesh_attn {
namespace host {

// Records printf-style text as the calling thread's last error; returns st.
ma_status_t fail(ma_status_t st, const char* fmt, ...)
    __attribute__((format(printf, 2, 3)));

// Clears the calling thread's last error; returns MA_OK.
ma_status_t ok();

}  // namespace host
}  // namespace mesh_attn
