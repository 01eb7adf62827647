// status.hpp -- the library's per-thread error message, shared by its translation units.
#pragma once

#include <string>

namespace treeens {

// Record the message tree_ens_last_error() returns on this thread; returns `code`.
int set_error(int code, const std::string &message);
// Clear it (every entry point starts with this).
void clear_error();

} // namespace treeens
