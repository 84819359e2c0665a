// The float32 Jacobian kernel compiled for fixed (n_max, l_max + 1) pairs:
// with the basis dimensions known to the compiler, its index arithmetic and
// loop bounds fold into constants.  Built once per part (JF_PART = 0, 1, 2)
// so the parts compile in parallel; each part answers for its n_max values.
#include "soap_device.h"

#ifndef JF_PART
#error "JF_PART must be defined"
#endif

#define JF_CAT2(a, b) a##b
#define JF_CAT(a, b) JF_CAT2(a, b)

namespace soap {

#define JF_CASE(N, LW)                                                                                             \
    if (n == N && lw == LW) return reinterpret_cast<const void *>(&dev::k_jacobian<float, float, N, LW>);
#define JF_ROW(N) JF_CASE(N, 3) JF_CASE(N, 5) JF_CASE(N, 7) JF_CASE(N, 9) JF_CASE(N, 11) JF_CASE(N, 13)

const void *JF_CAT(jacobian_fixed_, JF_PART)(int n, int lw) {
#if JF_PART == 0
    JF_ROW(2) JF_ROW(4)
#elif JF_PART == 1
    JF_ROW(6) JF_ROW(8)
#else
    JF_ROW(10) JF_ROW(12)
#endif
    return nullptr;
}

} // namespace soap
