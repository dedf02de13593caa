// Hooks the runtime (pipeline, checkpoint) uses beyond the public C ABI.
#pragma once
#include <string>

#include "../../include/zl.h"

namespace zl {
zl_status set_error(zl_status s, const std::string& msg);  // sets zl_last_error()
bool chunk_at_boundary(const zl_chunk* c);  // no call pending and no unapplied gradient
void chunk_close_window(zl_chunk* c);       // next backward overwrites the gradient
}  // namespace zl
