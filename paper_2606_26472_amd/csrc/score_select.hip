// The selection and the hidden-state scoring of one eviction step in a
// single launch, for chunks no longer than the recency window (C <= R).
// Then every new token lies in the protected window [N-R, N), so which of
// the older positions survive depends only on their frozen scores (Sec. 3.3)
// and not on the chunk being scored: the two are independent and can run
// side by side instead of one after the other.
//
// Workgroups [0, B) are the select kernel's (one sequence each); the rest
// carry 16 score wavefronts each (each wavefront one (sequence, layer,
// segment) unit, barrier-free).  Both run the very code of their own
// kernels (select_impl.h, score_hs_impl.h), so the results are those of the
// separate launches bit for bit.
#include "score_hs_impl.h"
#include "select_impl.h"

namespace epikv {
namespace {

constexpr int kUnitsPerBlock = kSelectThreads / 64;

template <int KPT, int VPW, int U>
__global__ __launch_bounds__(kSelectThreads) void k_select_score(SelectArgs sel, ScoreHsArgs sc) {
  if ((int)blockIdx.x < sel.B) {
    select_impl::select_seq<KPT>(sel, blockIdx.x);
    return;
  }
  const int64_t unit = (int64_t)(blockIdx.x - sel.B) * kUnitsPerBlock + (threadIdx.x >> 6);
  if (unit >= score_impl::wave_units(sc)) return;
  score_impl::score_hs_unit<VPW, U>(sc, (int)unit, threadIdx.x & 63);
}

template <int KPT, int VPW, int U>
hipError_t launch(const SelectArgs& sel, const ScoreHsArgs& sc, hipStream_t s) {
  const int64_t units = score_impl::wave_units(sc);
  const int64_t blocks = sel.B + (units + kUnitsPerBlock - 1) / kUnitsPerBlock;
  hipLaunchKernelGGL((k_select_score<KPT, VPW, U>), dim3((unsigned)blocks), dim3(kSelectThreads), 0,
                     s, sel, sc);
  return hipGetLastError();
}

template <int KPT>
hipError_t launch_vpw(const SelectArgs& sel, const ScoreHsArgs& sc, hipStream_t s) {
  // rows in flight chosen to stay within 128 registers (1024-thread blocks)
  const int nvec = sc.D / 8;
  if (nvec <= 64) return launch<KPT, 1, 8>(sel, sc, s);
  if (nvec <= 128) return launch<KPT, 2, 4>(sel, sc, s);
  if (nvec <= 256) return launch<KPT, 4, 2>(sel, sc, s);
  return launch<KPT, 8, 1>(sel, sc, s);
}

}  // namespace

bool select_score_fusable(const SelectArgs& sel, const ScoreHsArgs& sc) {
  return sc.C <= sel.R && sc.D / 8 <= 64 * 8;
}

hipError_t launch_select_score(const SelectArgs& sel, const ScoreHsArgs& score, hipStream_t s) {
  ScoreHsArgs sc = score;
  sc.seg_len = score_impl::wave_seg_len(sc);
  const int64_t per = (sel.ld_s + kSelectThreads - 1) / kSelectThreads;
  if (per <= 1) return launch_vpw<1>(sel, sc, s);
  if (per <= 2) return launch_vpw<2>(sel, sc, s);
  if (per <= 4) return launch_vpw<4>(sel, sc, s);
  if (per <= 8) return launch_vpw<8>(sel, sc, s);
  if (per <= 16) return launch_vpw<16>(sel, sc, s);
  if (per <= 32) return launch_vpw<32>(sel, sc, s);
  return launch_vpw<0>(sel, sc, s);
}

}  // namespace epikv
