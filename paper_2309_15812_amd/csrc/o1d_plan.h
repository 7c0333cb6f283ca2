// Device limits shared by the host-side plans of every kernel family.
#pragma once

#include <stddef.h>

namespace o1d {

constexpr int kThreads = 256;
constexpr size_t kMaxLdsBytes = 160 * 1024;  // gfx950 LDS per workgroup

}  // namespace o1d
