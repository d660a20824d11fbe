// Compile-time loop expansion shared by the kernel families.
#pragma once

#include <type_traits>
#include <utility>

namespace xtc {

// Calls f(std::integral_constant<int, I>()) for I = 0, 1, ...: a loop whose
// index is a compile-time constant in the body, however large the body (the
// compiler's unroller gives up on long bodies, and then register arrays
// indexed by the loop variable turn into indexed register moves).
template <typename F, int... I>
__device__ __forceinline__ void each_index(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>()), ...);
}

}  // namespace xtc
