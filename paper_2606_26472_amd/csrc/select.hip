// The selection kernel: one 1024-thread workgroup per sequence running
// select_seq (select_impl.h, which describes the method).
#include "select_impl.h"

namespace epikv {
namespace {

template <int KPT>
__global__ __launch_bounds__(kSelectThreads) void k_select(SelectArgs a) {
  select_impl::select_seq<KPT>(a, blockIdx.x);
}

template <int KPT>
hipError_t launch(const SelectArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_select<KPT>), dim3(a.B), dim3(kSelectThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  // Registers per thread for the keys: the smallest power of two covering
  // ld_s positions (every N is at most ld_s); beyond 32 per thread the keys
  // would spill, so longer rows take the global-memory variant.
  const int64_t per = (a.ld_s + kSelectThreads - 1) / kSelectThreads;
  if (per <= 1) return launch<1>(a, s);
  if (per <= 2) return launch<2>(a, s);
  if (per <= 4) return launch<4>(a, s);
  if (per <= 8) return launch<8>(a, s);
  if (per <= 16) return launch<16>(a, s);
  if (per <= 32) return launch<32>(a, s);
  return launch<0>(a, s);
}

}  // namespace epikv
