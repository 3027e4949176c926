// The eviction step's selection with one sequence split over G workgroups,
// for batches that would leave most of the device idle with one workgroup
// per sequence (a single long prefill, a small decode batch).
//
// What is selected is exactly what select_impl.h computes (Sec. 3.1,
// Sec. 3.3, App. D: the prefill, the recency window and the M = K-P-R best
// positions in between, ties to the lower position, ascending output); so
// is the method, a three-pass radix select of the M-th largest ranking key
// over 11/11/10-bit digits followed by an ordered write-out.  What changes
// is who does it: workgroup g of a sequence covers the positions
// [g*S, (g+1)*S), S = KPT * 1024, thread t holding the keys of positions
// g*S + k*1024 + t (k < KPT, so that every load is one contiguous row per
// wavefront), and the workgroups exchange counts through global memory:
//   pass p   each workgroup histograms its keys in LDS and adds the bins it
//            saw to the sequence's histogram for that pass (device-scope
//            atomics), then reads the whole histogram until it is complete
//            and takes the same digit decision as every other workgroup;
//   output   each workgroup publishes how many of its positions are kept
//            outright (outside the scored range, or a key above the
//            threshold T) and how many keys equal T, waits for all those
//            counts, and sums the ones of the workgroups before it: that
//            gives its first output slot and how many ties precede its own.
//            Inside the workgroup, positions are ranked in order by
//            wavefront ballots per row of 1024 and a prefix over the
//            (row, wavefront) counts, so the slots come out ascending and
//            ties are kept lowest position first, as with one workgroup.
//
// No barrier counter is needed: the totals are known in advance (pass 0
// counts every scored key plus one per workgroup; pass p+1 the keys in the
// digit pass p chose; the output counts add up to K - need kept outright
// and to the number of keys equal to T), and since every shared word starts
// at zero and only grows towards its final value, a read whose words add up
// to the known total has every word final.
//
// Each sequence's scratch therefore has to be clear when the kernel starts.
// A small fill kernel launched just before it writes every sequence's block
// (histograms and flags zero, a 64-bit marker that the block is clear), so
// nothing depends on what the workspace held before: it may have served
// another batch size's layout, or other data, since the previous call.
// (Each workgroup also zeroes its own count slot when it starts and its
// share of the histograms once every workgroup is past them; and a block
// found without the marker is cleared by the sequence's last workgroup,
// which then sets it, while the others wait.)
//
// The launcher keeps the grid within one workgroup per compute unit, so all
// of a sequence's workgroups can run together; should they not (other work
// holding the device), a waiting workgroup gives up after about a second,
// the sequence is flagged EPIKV_SEQ_SYNC and every wave still ends.
#include <atomic>

#include "select_impl.h"

namespace epikv {
namespace {

using select_impl::rank_key;

constexpr int kWaves = kSelectThreads / 64;
constexpr uint32_t kSpinLimit = 1u << 20;  // looks at the shared data before giving up (~1 s)

// Device-scope atomic accesses: every value that crosses workgroups (the
// histogram bins, the join count, the per-workgroup counts) is written and
// read only through these, which the hardware keeps coherent across the
// whole device without cache maintenance.
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void add_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_or_zero(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// Inclusive prefix sum over the 64 lanes of a wavefront: shifts of 1, 2, 4
// and 8 lanes inside each row of 16, then the row totals.
__device__ __forceinline__ uint32_t wave_scan(uint32_t v) {
  v += dpp_or_zero<0x111>(v);  // row_shr:1
  v += dpp_or_zero<0x112>(v);  // row_shr:2
  v += dpp_or_zero<0x114>(v);  // row_shr:4
  v += dpp_or_zero<0x118>(v);  // row_shr:8
  const uint32_t r0 = __builtin_amdgcn_readlane(v, 15);
  const uint32_t r1 = __builtin_amdgcn_readlane(v, 31);
  const uint32_t r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return v + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Set bits of m in the lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Sum of v over the workgroup, the same in every thread (wtot: kWaves words
// of LDS).  One barrier: callers alternate between two wtot buffers, so a
// buffer is rewritten only after the barrier of the call in between.
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* wtot) {
  const int wave = threadIdx.x >> 6;
  v = wave_scan(v);
  if ((threadIdx.x & 63) == 63) wtot[wave] = v;
  __syncthreads();
  uint32_t t = 0u;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t += wtot[w];
  return t;
}

// Wavefront 0, on a table of n <= 4 * 64 counts in LDS: replace each by the
// sum of the ones before it and return the total.  Lane l takes the entries
// [4l, 4l + 4).
__device__ __forceinline__ uint32_t wave_exclusive_table(uint32_t* tab, int n) {
  const int lane = threadIdx.x & 63;
  uint32_t v[4];
  uint32_t local = 0u;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * lane + j;
    v[j] = e < n ? tab[e] : 0u;
    local += v[j];
  }
  const uint32_t incl = wave_scan(local);
  uint32_t run = incl - local;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * lane + j;
    if (e < n) tab[e] = run;
    run += v[j];
  }
  return __builtin_amdgcn_readlane(incl, 63);
}

// The sequence's scratch carries the marker that it is clear.
__device__ __forceinline__ bool marked(const uint32_t* seq) {
  return ld_dev(&seq[0]) == kSelMarkLo && ld_dev(&seq[1]) == kSelMarkHi;
}

// Mark the sequence as given up: its scratch as not clear (the next call
// clears it), the give-up flag raised, and the status.  (A workgroup that
// gives up while waiting for a histogram never contributes to the next
// step, so no other workgroup of the sequence can complete.)
__device__ __forceinline__ void give_up(const SelectArgs& a, int b, uint32_t* seq) {
  if (threadIdx.x == 0) {
    __hip_atomic_store(&seq[0], 0u, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_AGENT);  // not clear
    __hip_atomic_store(&seq[2], 1u, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_AGENT);
    a.n_keep[b] = -1;
    a.seq_status[b] = EPIKV_SEQ_SYNC;
  }
}

// Wavefront 0: the digit holding the need-th largest key of the histogram
// of NB bins in hist (16-byte aligned).  Lane l sums the bins
// [NB - (l+1)*BPL, NB - l*BPL) (so the lanes run over descending digits),
// reading them 16 bytes at a time in a rotated order that spreads the LDS
// banks; a wavefront scan finds the lane whose bins hold the need-th key; a
// second scan over that lane's bins, one per lane, finds the bin.
// out[0] = the digit, out[1] = keys in higher digits, out[2] = keys in it.
template <int NB>
__device__ __forceinline__ void find_digit_wave(const uint32_t* hist, uint32_t need,
                                                uint32_t* out) {
  constexpr int kBpl = NB / 64;
  constexpr int kVec = kBpl / 4;
  const int lane = threadIdx.x & 63;
  const uint4* v = reinterpret_cast<const uint4*>(hist + (NB - (lane + 1) * kBpl));
  uint32_t local = 0u;
#pragma unroll
  for (int j = 0; j < kVec; ++j) {
    const uint4 x = v[(j + lane) & (kVec - 1)];
    local += x.x + x.y + x.z + x.w;
  }
  const uint32_t incl = wave_scan(local);
  const uint32_t excl = incl - local;
  const uint64_t hit = __ballot(excl < need && need <= incl);
  const int L = hit ? __ffsll((unsigned long long)hit) - 1 : 0;
  const uint32_t ex_l = __builtin_amdgcn_readlane(excl, L);
  const int top_l = NB - 1 - L * kBpl;
  const uint32_t h = lane < kBpl ? hist[top_l - lane] : 0u;
  const uint32_t in2 = wave_scan(h) + ex_l;
  const uint32_t ex2 = in2 - h;
  const uint64_t hit2 = __ballot(lane < kBpl && ex2 < need && need <= in2);
  const int q = hit2 ? __ffsll((unsigned long long)hit2) - 1 : 0;
  if (lane == q) {
    out[0] = (uint32_t)(top_l - q);
    out[1] = ex2;
    out[2] = h;
  }
}

template <int KPT>
__global__ __launch_bounds__(kSelectThreads) void k_select_multi(SelectMultiArgs m) {
  __shared__ __align__(16) uint32_t hist[2048];
  __shared__ uint32_t tab[2][KPT * kWaves];  // per (row of 1024, wavefront) counts
  __shared__ uint32_t wtot[2][kWaves];
  __shared__ uint32_t bcast[8];
  const SelectArgs& a = m.sel;
  const int G = m.groups;
  const int b = (int)blockIdx.x / G;
  const int g = (int)blockIdx.x - b * G;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  constexpr int kSpan = KPT * kSelectThreads;
  const int g0 = g * kSpan;  // first position of this workgroup's slice
  // The slice's scores are loaded first: their addresses do not depend on
  // the sequence's counts, so the two loads are in flight together.
  const float* s = a.scores + (int64_t)b * a.ld_s;
  float raw[KPT];
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const int i = g0 + k * kSelectThreads + tid;
    raw[k] = i < a.ld_s ? s[i] : 0.f;
  }
  const int N = a.n_cached[b];
  const int P = a.n_prefix[b];
  const int K = a.K;
  const int R = a.R;
  int32_t* out = a.keep_idx + (int64_t)b * K;

  // Decisions that end a sequence early are the same in all its workgroups,
  // so none of them is left waiting for the others.
  if (N < a.min_n || (int64_t)N > a.ld_s || P < 0) {
    if (g == 0 && tid == 0) {
      a.n_keep[b] = -1;
      a.seq_status[b] = EPIKV_SEQ_RANGE;
    }
    return;
  }
  if (N <= K) {
    const int end = min(N, g0 + kSpan);
    for (int j = g0 + tid; j < end; j += kSelectThreads) out[j] = j;
    if (g == 0 && tid == 0) {
      a.n_keep[b] = N;
      a.seq_status[b] = EPIKV_SEQ_OK;
    }
    return;
  }
  if ((int64_t)P + R >= K) {
    if (g == 0 && tid == 0) {
      a.n_keep[b] = -1;
      a.seq_status[b] = EPIKV_SEQ_BUDGET;
    }
    return;
  }

  // (the look at the marker overlaps the scores' loads)
  const int lo = P, hi = N - R;  // eligible positions [lo, hi)
  uint32_t keys[KPT];
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const int i = g0 + k * kSelectThreads + tid;
    keys[k] = (i >= lo && i < hi) ? rank_key(raw[k]) : 0u;
  }

  uint32_t* seq = m.scratch + (size_t)b * kSelSeqWords;
  uint32_t* gave_up = seq + 2;
  uint32_t* joined = seq + 3;                                // workgroups that started
  uint32_t* ghist = seq + kSelHeadWords;                     // [3][2048]
  uint32_t* counts = m.scratch + (size_t)a.B * kSelSeqWords;  // [B*G][2]
  if (tid == 0) bcast[0] = marked(seq) ? 1u : 0u;
  __syncthreads();
  if (!bcast[0]) {
    if (g == G - 1) {
      // Not known to be clear: this workgroup clears it and sets the
      // marker (its high word first, so that a reader seeing the low word
      // sees both); the others wait for the marker.
      for (int i = tid; i < 3 * 2048; i += kSelectThreads) st_dev(&ghist[i], 0u);
      if (tid == 0) {
        st_dev(gave_up, 0u);
        st_dev(joined, 0u);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0) {
        st_dev(&seq[1], kSelMarkHi);
        __builtin_amdgcn_s_waitcnt(0);
        st_dev(&seq[0], kSelMarkLo);
      }
    } else {
      if (tid == 0) {
        uint32_t spins = 0;
        while (!marked(seq) && spins < kSpinLimit) {
          __builtin_amdgcn_s_sleep(1);
          ++spins;
        }
        bcast[1] = marked(seq) ? 1u : 0u;
      }
      __syncthreads();
      if (!bcast[1]) {
        give_up(a, b, seq);
        return;
      }
    }
  }
  __syncthreads();  // bcast is rewritten
  if (tid == 0) {
    st_dev(&counts[2 * (size_t)blockIdx.x], 0u);
    st_dev(&counts[2 * (size_t)blockIdx.x + 1], 0u);
  }

  uint32_t prefix = 0u, mask = 0u;
  uint32_t need = (uint32_t)(K - P - R);  // rank (1-based) of the threshold key
  // what the pass's histogram will hold: in pass 0 every scored key, and
  // the workgroups that joined (each zeroed its count slot first)
  uint32_t expect = (uint32_t)(hi - lo) + (uint32_t)G;
#pragma unroll 1
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : pass == 1 ? 10 : 0;
    const int nb = pass == 2 ? 1024 : 2048;
    const uint32_t dmask = (uint32_t)nb - 1u;
    uint32_t* gh = ghist + pass * 2048;
    for (int i = tid; i < nb; i += kSelectThreads) hist[i] = 0u;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int i = g0 + k * kSelectThreads + tid;
      if (i >= lo && i < hi && (keys[k] & mask) == prefix)
        atomicAdd(&hist[(keys[k] >> shift) & dmask], 1u);
    }
    __syncthreads();
    if (pass == 0) {
      __builtin_amdgcn_s_waitcnt(0);  // the count slot's zeroing is done
      if (tid == 0) add_dev(joined, 1u);
    }
    for (int i = tid; i < nb; i += kSelectThreads) {
      const uint32_t h = hist[i];
      if (h) add_dev(&gh[i], h);
    }
    // Wait for the other workgroups' bins: the bins only grow, from zero,
    // and in the end hold exactly `expect`, so a read whose bins add up to
    // `expect` has every bin final.
    for (uint32_t spins = 0;; ++spins) {
      uint32_t part = (pass == 0 && tid == 0) ? ld_dev(joined) : 0u;
      for (int i = tid; i < nb; i += kSelectThreads) {
        const uint32_t h = ld_dev(&gh[i]);
        hist[i] = h;
        part += h;
      }
      if (block_sum(part, wtot[spins & 1]) == expect) break;
      if (spins == kSpinLimit) {
        give_up(a, b, seq);
        return;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (tid < 64) {
      if (pass == 2)
        find_digit_wave<1024>(hist, need, bcast);
      else
        find_digit_wave<2048>(hist, need, bcast);
    }
    __syncthreads();
    prefix |= bcast[0] << shift;
    mask |= dmask << shift;
    need -= bcast[1];
    expect = bcast[2];
    // (bcast is next written by the next pass's search, barriers later)
  }

  // need = keys equal to T that are kept, lowest positions first; expect =
  // keys equal to T.  Per (row k, wavefront): keys equal to T, and
  // positions kept outright.
  const uint32_t T = prefix;
  constexpr int kTab = KPT * kWaves;
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const int i = g0 + k * kSelectThreads + tid;
    const bool elig = i >= lo && i < hi;
    const uint64_t m_eq = __ballot(elig && keys[k] == T);
    const uint64_t m_out = __ballot(i < N && (!elig || keys[k] > T));
    if (lane == 0) {
      tab[0][k * kWaves + wave] = (uint32_t)__popcll(m_eq);
      tab[1][k * kWaves + wave] = (uint32_t)__popcll(m_out);
    }
  }
  __syncthreads();
  // Wavefront 0: ranks of the ties before each (row, wavefront), this
  // workgroup's counts published, then those of all workgroups of the
  // sequence waited for -- kept outright (the P + R protected positions and
  // the keys above T, K - need in all) and equal to T (expect in all);
  // written once each, from zero, so reads that add up to both totals are
  // final -- and the ones before this workgroup summed (G <= kSelMaxGrid).
  if (tid < 64) {
    const uint32_t eq_tot = wave_exclusive_table(tab[0], kTab);
    const uint32_t out_tot = wave_exclusive_table(tab[1], kTab);
    if (lane == 0) {
      st_dev(&counts[2 * (size_t)blockIdx.x], out_tot);
      st_dev(&counts[2 * (size_t)blockIdx.x + 1], eq_tot);
    }
    const uint32_t want_out = (uint32_t)K - need, want_eq = expect;
    uint32_t c_out = 0u, c_eq = 0u, done = 0u;
    for (uint32_t spins = 0;; ++spins) {
      uint32_t t_out = 0u, t_eq = 0u;
      c_out = 0u;
      c_eq = 0u;
      for (int w = lane; w < G; w += 64) {
        const size_t x = (size_t)b * G + w;
        const uint32_t o = ld_dev(&counts[2 * x]);
        const uint32_t e = ld_dev(&counts[2 * x + 1]);
        t_out += o;
        t_eq += e;
        c_out += w < g ? o : 0u;
        c_eq += w < g ? e : 0u;
      }
      t_out = __builtin_amdgcn_readlane(wave_scan(t_out), 63);
      t_eq = __builtin_amdgcn_readlane(wave_scan(t_eq), 63);
      if (t_out == want_out && t_eq == want_eq) {
        done = 1u;
        break;
      }
      // Giving up here, the flag is raised before one last look, so that
      // the workgroup writing the status -- which can still see all counts
      // later -- is sure to see the flag too.
      if (spins == kSpinLimit + 1) break;
      if (spins == kSpinLimit && lane == 0)
        __hip_atomic_store(gave_up, 1u, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_sleep(1);
    }
    c_out = wave_scan(c_out);
    c_eq = wave_scan(c_eq);
    if (lane == 63) {
      bcast[0] = c_out;
      bcast[1] = c_eq;
      bcast[2] = done;
    }
  }
  __syncthreads();
  if (!bcast[2]) {
    give_up(a, b, seq);
    return;
  }
  // Every workgroup has published its counts, so none reads the histograms
  // or the join count again: clear this workgroup's share for the next call.
  {
    const int per = (3 * 2048 + G - 1) / G;
    const int end = min(3 * 2048, (g + 1) * per);
    for (int i = g * per + tid; i < end; i += kSelectThreads) st_dev(&ghist[i], 0u);
    if (g == 0 && tid == 0) st_dev(joined, 0u);
  }
  const uint32_t out_before = bcast[0], eq_before = bcast[1];
  const uint32_t kept_before = out_before + min(need, eq_before);

  // Which positions are kept: a tie is kept while its rank among the
  // sequence's ties (in position order) is below need.
  uint32_t keep_bits = 0u;
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const int i = g0 + k * kSelectThreads + tid;
    const bool elig = i >= lo && i < hi;
    const bool eq = elig && keys[k] == T;
    const uint64_t m_eq = __ballot(eq);
    const uint32_t rank = eq_before + tab[0][k * kWaves + wave] + lanes_below(m_eq);
    const bool keep = i < N && (!elig || keys[k] > T || (eq && rank < need));
    keep_bits |= keep ? 1u << k : 0u;
    const uint64_t m_keep = __ballot(keep);
    if (lane == 0) tab[1][k * kWaves + wave] = (uint32_t)__popcll(m_keep);
  }
  __syncthreads();
  if (tid < 64) {
    const uint32_t kept_here = wave_exclusive_table(tab[1], kTab);
    if (lane == 0) bcast[3] = kept_here;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const bool keep = (keep_bits >> k) & 1u;
    const uint64_t m_keep = __ballot(keep);
    const uint32_t slot = kept_before + tab[1][k * kWaves + wave] + lanes_below(m_keep);
    if (keep && slot < (uint32_t)K) out[slot] = g0 + k * kSelectThreads + tid;
  }
  if (g == G - 1 && tid == 0) {
    // A workgroup that gave up set the flag before its last look at the
    // counts, which then still missed some; this one saw them all
    // afterwards, so the flag is visible here.
    const bool sync_ok =
        __hip_atomic_load(gave_up, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_AGENT) == 0u;
    const bool ok_k = kept_before + bcast[3] == (uint32_t)K;
    a.n_keep[b] = (sync_ok && ok_k) ? K : -1;
    a.seq_status[b] = !sync_ok ? EPIKV_SEQ_SYNC : ok_k ? EPIKV_SEQ_OK : EPIKV_SEQ_RANGE;
  }
}

template <int KPT>
hipError_t launch(const SelectMultiArgs& m, hipStream_t s) {
  hipLaunchKernelGGL((k_select_multi<KPT>), dim3((unsigned)(m.sel.B * m.groups)),
                     dim3(kSelectThreads), 0, s, m);
  return hipGetLastError();
}

// Compute units of the current device (0 if the query fails), looked up
// once per device.  The grid is kept within one workgroup per unit: that is
// always resident, and measured faster than sharing units between two.
int device_cus() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v <= 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

constexpr size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Every sequence's scratch block made clear before the selection: head
// words zero but for the marker, histograms zero.  One thread per word of
// the first n_words words (the B sequences' blocks).
__global__ __launch_bounds__(256) void k_select_scratch_clear(uint32_t* scratch, int64_t n_words) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_words) return;
  const int64_t w = i % kSelSeqWords;
  scratch[i] = w == 0 ? kSelMarkLo : (w == 1 ? kSelMarkHi : 0u);
}

}  // namespace

size_t select_scratch_bytes(int B) {
  if (B < 1 || 2 * B > kSelMaxGrid) return 0;  // never split: at most one workgroup each
  return align256((size_t)B * kSelSeqWords * 4 + (size_t)kSelMaxGrid * 8);
}

hipError_t launch_select_groups(const SelectArgs& a, void* scratch, hipStream_t s) {
  // The fewest keys per thread (1, 2, 4, 8 or 16; 32 would spill) whose
  // grid fits one workgroup per compute unit, so that a sequence's
  // workgroups all run together.
  int v = -1, groups = 1;
  const int64_t cap = min(kSelMaxGrid, device_cus());
  if (scratch && select_scratch_bytes(a.B) > 0) {
    for (int j = 0; j < 5; ++j) {
      const int64_t span = (int64_t)(1 << j) * kSelectThreads;
      const int64_t G = (a.ld_s + span - 1) / span;
      if (G < 2) break;  // one workgroup covers the row: nothing to split
      if ((int64_t)a.B * G <= cap) {
        v = j;
        groups = (int)G;
        break;
      }
    }
  }
  if (v < 0) return launch_select(a, s);

  // The scratch is cleared here rather than trusted to be as the previous
  // call left it: a workspace may have held other data since (another
  // batch size's layout, or the caller's own use), and a stale count would
  // leave a histogram that never adds up.
  const int64_t n_words = (int64_t)a.B * kSelSeqWords;
  hipLaunchKernelGGL(k_select_scratch_clear, dim3((unsigned)((n_words + 255) / 256)), dim3(256), 0, s,
                     (uint32_t*)scratch, n_words);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  SelectMultiArgs m;
  m.sel = a;
  m.scratch = (uint32_t*)scratch;
  m.groups = groups;
  switch (v) {
    case 0: return launch<1>(m, s);
    case 1: return launch<2>(m, s);
    case 2: return launch<4>(m, s);
    case 3: return launch<8>(m, s);
    default: return launch<16>(m, s);
  }
}

}  // namespace epikv
