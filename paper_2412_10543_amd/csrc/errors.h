// Error reporting shared by the C ABI's source files (internal): the
// thread-local message behind rag_last_error().
#pragma once

#include "rag_attn.h"

namespace rag {

// Sets the message (printf-style) and returns st.
rag_status fail(rag_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clears the message and returns RAG_OK.
rag_status ok();

}  // namespace rag
