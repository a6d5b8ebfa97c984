// Host-side helpers shared by the launchers.
#include <mutex>
#include <unordered_map>

#include "common.h"

namespace dqn {

// Raise a kernel's dynamic LDS limit to the largest size it is launched
// with (once per kernel and size; thread-safe).
bool allow_lds(const void* kern, size_t bytes) {
    static std::mutex mu;
    static std::unordered_map<const void*, size_t> granted;
    std::lock_guard<std::mutex> lock(mu);
    size_t& g = granted[kern];
    if (bytes <= g) return true;
    if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) != hipSuccess)
        return false;
    g = bytes;
    return true;
}

}  // namespace dqn
