// amsim_tab.hip -- the table kernels of one operation, AMSIM_TAB_OP (0 GEMM, 1 forward,
// 2 backward data, 3 backward weight; set by the build, which compiles this file once per
// operation so that the four instantiation sets build in parallel), with their launch and
// attribute set-up.
#include "amsim_tab.h"

#ifndef AMSIM_TAB_OP
#error "AMSIM_TAB_OP must name the operation (0..3)"
#endif

namespace amsim_detail __attribute__((visibility("hidden"))) {

namespace {

// Raises the kernel's dynamic LDS limit, and checks that it has no static LDS: the bf16 path
// addresses its slabs as LDS addresses starting at 0.  Keeps the first error in err.
template <typename K>
void allow_lds(K kernel, size_t bytes, hipError_t &err)
{
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
    hipFuncAttributes fa{};
    if (e == hipSuccess) e = hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(kernel));
    if (e == hipSuccess && fa.sharedSizeBytes != 0) e = hipErrorInvalidKernelFile;
    if (err == hipSuccess) err = e;
}

template <typename F>
void dispatch_tab_tile(const Tile &t, int rl, F &&f)
{
#define X(TM, TN, WR, NW, RL)                                                             \
    if (t.tm == TM && t.tn == TN && t.wr == WR && t.nw == NW && rl == RL) {               \
        f(std::integral_constant<int, TM>{}, std::integral_constant<int, TN>{},           \
          std::integral_constant<int, WR>{}, std::integral_constant<int, NW>{},           \
          std::integral_constant<int, RL>{});                                             \
        return;                                                                           \
    }
    AMSIM_FOR_TAB_TILES(X)
#undef X
}

}  // namespace

template <int OP>
hipError_t tab_attributes()
{
    hipError_t err = hipSuccess;
#define X(TM, TN, WR, NW, RL)                                                                              \
    allow_lds(tab_kernel<OP, TM, TN, WR, NW, RL, kTabApprox>, tab_lds_bytes(TN, WR, NW, RL), err);          \
    if constexpr (RL == 7) {                                                                                \
        allow_lds(tab_kernel<OP, TM, TN, WR, NW, 7, kTabNative>, tab_native_lds_bytes(TN, WR, NW), err);    \
        allow_lds(tab_kernel<OP, TM, TN, WR, NW, 7, kTabApproxSelf>, tab_lds_bytes(TN, WR, NW, 7), err);    \
    }
    AMSIM_FOR_TAB_TILES(X)
#undef X
    return err;
}

template <int OP>
hipError_t tab_launch(const Tile &t, int rl, int var, const TabArgs &a, dim3 grid, hipStream_t st)
{
    bool launched = false;
    auto run = [&](auto tm, auto tn, auto wr, auto nw, auto rl_c) {
        constexpr int TM = decltype(tm)::value, TN = decltype(tn)::value, WR = decltype(wr)::value;
        constexpr int NW = decltype(nw)::value, RL = decltype(rl_c)::value;
        if (var == kTabNative) {
            if constexpr (RL == 7) {
                hipLaunchKernelGGL((tab_kernel<OP, TM, TN, WR, NW, 7, kTabNative>), grid, dim3(64 * NW),
                                   tab_native_lds_bytes(TN, WR, NW), st, a);
                launched = true;
            }
            return;
        }
        if (var == kTabApproxSelf) {  // rows of 128 entries only
            if constexpr (RL == 7) {
                hipLaunchKernelGGL((tab_kernel<OP, TM, TN, WR, NW, 7, kTabApproxSelf>), grid, dim3(64 * NW),
                                   tab_lds_bytes(TN, WR, NW, 7), st, a);
                launched = true;
            }
            return;
        }
        hipLaunchKernelGGL((tab_kernel<OP, TM, TN, WR, NW, RL, kTabApprox>), grid, dim3(64 * NW),
                           tab_lds_bytes(TN, WR, NW, RL), st, a);
        launched = true;
    };
    dispatch_tab_tile(t, rl, run);
    return launched ? hipGetLastError() : hipErrorInvalidConfiguration;
}

template hipError_t tab_attributes<AMSIM_TAB_OP>();
template hipError_t tab_launch<AMSIM_TAB_OP>(const Tile &, int, int, const TabArgs &, dim3, hipStream_t);

}  // namespace amsim_detail
