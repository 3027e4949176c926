// KV-vector signals, Sec. 3.3 and Table 1:
//   Lag-KV      x~ = (x - mn) / (mx - mn + eps) per channel, with (mn, mx) the
//               range of the previous chunk at the same (layer, K|V, head,
//               channel), for keys and values;
//   lag-kv-key  the same, keys only;
//   KV-key/val  x~ = x, keys (values) only;
//   v(t, l, kv, h) = population variance of x~ over the head dimension;
//   q(t) = mean over (layer, head) of the sum of v over the used tensors.
// For the lag-normalised signals the chunk's own per-channel range is written
// out as the next chunk's reference; the first chunk of a stream, with no
// previous chunk, is normalised by its own range.
//
// Kernel 1: one workgroup per (sequence, used plane) -- a plane is one
// (layer, K|V) of a used tensor, so signals of one tensor launch half as
// many -- streaming the chunk's rows of that plane from the paged pool:
// 512 threads for the lag-normalised signals (four registers of state per
// channel), 1024 for the raw ones.  When that gives too few workgroups to
// fill the GPU the rows are split between `splits` workgroups, whose
// partial channel ranges the second kernel combines; otherwise the
// workgroup writes the chunk's range itself.
// A lane owns one 16-byte column = 8 channels of one head.  A wavefront
// takes a segment of 512 channels of a row (rows of 1024 channels: two
// wavefronts per row, each writing its own partial sum), or several narrow
// rows; with row segments the row, its page and its address are
// wave-uniform (scalar): a wavefront walks its rows in blocks of 64 whose
// byte offsets sit one per lane (read from an LDS table of the
// workgroup's rows, computed once, when the chunk is short enough).  Each
// wavefront keeps a fixed number of rows in flight: the loads of the next
// rows are issued as soon as a pair of rows has been used, unconditionally
// (rows past its block are empty loads), so that every use waits for its
// own rows only.
//   Variance, one pass: the sum and the sum of squares over the head.  For
//   the lag-normalised signals each channel is mapped to
//   y = (x - mn) / (mx - mn + eps) - 1/2 (the shift keeps the sums of
//   squares free of cancellation; a variance does not change under a
//   shift); for the raw signals the packed bf16 words feed
//   v_dot2_f32_bf16 directly (x0 + x1 and x0^2 + x1^2 in one instruction
//   each, no unpacking).  Each lane's two sums of a row go to LDS; per
//   batch of rows a transposed pass gives each lane one (row, head) pair,
//   whose lanes' sums it adds in lane order, and the heads of a row are
//   added with DPP row operations -- a few instructions per row instead of
//   a cross-lane reduction of every row.
//   Range (lag-normalised, not the first chunk): IEEE minimum / maximum
//   over the rows -- a NaN propagates, as in a plain minimum over the chunk
//   -- with three-input instructions over pairs of rows; the row slots'
//   ranges meet in LDS, one slot each, and are reduced channel by channel
//   in slot order.
//   First chunk of a stream (lag-normalised): a first pass over the rows
//   finds the chunk's range, the second computes the variances with it.
// Per (row, plane, segment) the sum of its heads' variances goes to
// partial[b][plane][segment][c].
// Kernel 2 sums the planes in a fixed order and divides by L*H, and (split
// rows) combines the splits' channel ranges into the next chunk's reference.
#include "epikv_internal.h"

namespace epikv {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) int lds_int;
typedef __attribute__((address_space(3))) int64_t lds_i64;

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of `width` lanes (1..64); every lane of a group
// ends with the same bits (each step adds two values that the partner lane
// adds in the other order).  Within a row of 16 lanes: DPP moves (quad
// permutes, half-row mirror, rotations); across rows: lane shuffles.
__device__ __forceinline__ float group_sum(float v, int width) {
  if (width <= 1) return v;
  if (width == 2) return v + dpp<0xB1>(v);  // quad_perm [1,0,3,2]
  if (width == 4) {
    v += dpp<0xB1>(v);
    return v + dpp<0x4E>(v);                // quad_perm [2,3,0,1]
  }
  if (width == 8) {
    v += dpp<0x141>(v);  // row_half_mirror: lane i + lane 7-i
    v += dpp<0x4E>(v);
    return v + dpp<0xB1>(v);
  }
  v += dpp<0x128>(v);    // row_ror:8
  v += dpp<0x124>(v);    // row_ror:4
  v += dpp<0x122>(v);    // row_ror:2
  v += dpp<0x121>(v);    // row_ror:1
  if (width >= 32) v += __shfl_xor(v, 16, 64);
  if (width == 64) v += __shfl_xor(v, 32, 64);
  return v;
}

// Order of one wavefront's LDS accesses by its own lanes: the hardware
// keeps them in issue order, the compiler must not move them across this.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Transposed head reduction (rows spanning whole wavefronts): each lane's
// sum and sum of squares over its channels of a row go to LDS, the rows in
// flight of kRedRowWords per wavefront; the padding after every 8 lanes
// makes the transposed reads (8 lanes apart) hit distinct banks.
__device__ __forceinline__ int red_word(int lane) { return (lane >> 3) * 20 + (lane & 7) * 2; }

// NW consecutive 32-bit words (2 * NW bf16 channels, NW a multiple of 4)
// of a row whose address is wave-uniform: a buffer resource made for the
// row (scalar registers) and the lane's byte offset as the only vector
// operand, so a row costs no vector address arithmetic.  The resource
// spans the row alone; a missing row gets an empty resource, whose loads
// return 0 without a memory access.  Non-temporal: each byte is read once.
template <int NW>
__device__ __forceinline__ void ld_row_nt(const char* row, uint32_t off, int n_bytes,
                                          uint32_t (&w)[NW]) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)row, (short)0, n_bytes, kBufferRsrcWord3);
#pragma unroll
  for (int c = 0; c < NW / 4; ++c) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * c, 0, kBufferNonTemporal);
#pragma unroll
    for (int k = 0; k < 4; ++k) w[4 * c + k] = v[k];
  }
}
// The same through a per-lane address (rows narrower than a wavefront).
template <int NW>
__device__ __forceinline__ void ld_lane_nt(const char* p, uint32_t (&w)[NW]) {
#pragma unroll
  for (int c = 0; c < NW / 4; ++c) {
    const u32x4 v = ld_stream(p + 16 * c);
#pragma unroll
    for (int k = 0; k < 4; ++k) w[4 * c + k] = v[k];
  }
}

__device__ __forceinline__ float nan_min(float a, float b) {
  return __builtin_elementwise_minimum(a, b);
}
__device__ __forceinline__ float nan_max(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}

// LAG: lag-normalised signal.  NW: words (2 * NW channels) per lane.
// WIDE: rows of at least 64 lanes, split into segments of 64 lanes, one
// segment per wavefront, so the row, its page and its address are
// wave-uniform; narrower rows are shared by the lanes of one wavefront,
// 64 / (lanes per row) rows at a time.  WAVES: wavefronts per workgroup;
// AH: rows each keeps in flight.  The lag-normalised signals carry four
// registers of state per channel (the previous range's minimum and
// scale, the running minimum and maximum): 512-thread workgroups of up
// to 128 registers per lane with 8 rows in flight.  The raw signals carry
// none: 1024-thread workgroups within 64 registers (two per CU), 4 rows in
// flight.  RT (rows of whole wavefronts, chunks of up to kLagRowCache
// rows): the byte offsets of the workgroup's rows are computed once into
// LDS, so the loop over the rows holds none of the page-table arithmetic
// (which otherwise spills scalar registers).
template <bool LAG, bool WIDE, int NW, bool RT, bool BIG>
__global__ __launch_bounds__(lagkv_threads(LAG, BIG))
__attribute__((amdgpu_waves_per_eu(LAG ? 4 : 8))) void k_score_lagkv(ScoreLagArgs a) {
  constexpr int NCH = 2 * NW;               // channels per lane
  constexpr int WAVES = lagkv_waves(LAG, BIG);  // wavefronts per workgroup
  constexpr int NT = WAVES * 64;
  constexpr int AH = lagkv_ahead(LAG);      // rows in flight per wavefront
  extern __shared__ __align__(16) float lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int p = blockIdx.x;     // used plane
  const int b = blockIdx.y;
  const int sp = blockIdx.z;    // share of the chunk's rows
  const int layer = a.two ? p >> 1 : p;
  const int kv = a.two ? (p & 1) : a.kv0;
  const int HD = a.H * a.d;
  const int row_lanes = HD / NCH;                   // lanes per row
  const int segs = WIDE ? row_lanes / 64 : 1;       // wavefronts per row
  const int lpr = WIDE ? 64 : row_lanes;            // lanes per row segment
  const int rpw = WIDE ? 1 : 64 / row_lanes;        // rows per wavefront
  const int seg = WIDE ? wave % segs : 0;           // this wavefront's segment
  const int slot = WIDE ? wave / segs : wave;       // its row slot in the workgroup
  const int rw = WIDE ? 0 : lane / lpr;             // this lane's row within the wavefront's
  const int li = lane - rw * lpr;                   // lane within the segment
  const int col = seg * 64 + li;                    // this lane's group of NCH channels
  const int gw = a.d / NCH;                         // lanes per head
  const int row_bytes = HD * 2;

  const int N = a.n_cached[b];
  const int start = N - a.C;
  const bool seq_ok = start >= 0 && (int64_t)((N - 1) / a.page_size) < a.ld_pt;
  const int32_t* pt = a.pt + (int64_t)b * a.ld_pt;
  const int64_t half = (int64_t)a.B * a.L * 2 * HD;
  // this lane's first channel in the [2][B][L][2][H][d] range layout
  const int64_t rbase = (((int64_t)b * a.L + layer) * 2 + kv) * HD + col * NCH;
  const bool fresh = LAG && a.n_tok_in[b] <= 0;
  // The previous chunk's range of this lane's channels (carried state),
  // loaded first as whole vectors, so that its latency overlaps the set-up
  // of the row table instead of delaying the first rows.
  float rin[LAG ? 2 * NCH : 1];
  if (LAG && !fresh) {
    const float4* qmn = reinterpret_cast<const float4*>(a.range_in + rbase);
    const float4* qmx = reinterpret_cast<const float4*>(a.range_in + half + rbase);
#pragma unroll
    for (int k = 0; k < NCH / 4; ++k) {
      const float4 u = qmn[k], v = qmx[k];
      rin[4 * k] = u.x;
      rin[4 * k + 1] = u.y;
      rin[4 * k + 2] = u.z;
      rin[4 * k + 3] = u.w;
      rin[NCH + 4 * k] = v.x;
      rin[NCH + 4 * k + 1] = v.y;
      rin[NCH + 4 * k + 2] = v.z;
      rin[NCH + 4 * k + 3] = v.w;
    }
  }
  // this segment's row of partial sums [B][plane][segment][C]
  float* part = a.partial + (((int64_t)b * a.n_planes + p) * segs + seg) * a.C;

  // Rows [r_lo, r_hi) of the chunk are this workgroup's.  The first chunk
  // of a stream needs every row for its range before any variance: the
  // first share takes it whole.
  int r_lo = 0, r_hi = 0;
  if (fresh) {
    r_hi = sp == 0 ? a.C : 0;
  } else {
    const int per = (a.C + a.splits - 1) / a.splits;
    r_lo = min(a.C, sp * per);
    r_hi = min(a.C, r_lo + per);
  }
  const int slots = WAVES / segs;                         // row slots of the workgroup
  // Each row slot walks its own contiguous block of the share's rows, rpw
  // rows per sweep (narrow rows: one per lane group), so consecutive rows
  // of a wavefront mostly share a page.
  const int per_slot = ((r_hi - r_lo + slots - 1) / slots + rpw - 1) / rpw * rpw;
  const int s_lo = min(r_hi, r_lo + slot * per_slot);
  const int s_hi = min(r_hi, s_lo + per_slot);
  const int sweeps = (s_hi - s_lo + rpw - 1) / rpw;     // this wavefront's
  auto row_of = [&](int it) { return s_lo + it * rpw + rw; };
  // The share's rows are consecutive positions, so they need few pages:
  // their page-table entries are copied to LDS once (when they fit).
  auto page_index = [&](int pos) -> int {
    return a.page_shift >= 0 ? pos >> a.page_shift : pos / a.page_size;
  };
  const bool any_rows = seq_ok && r_hi > r_lo;
  const int pg0 = any_rows ? page_index(start + r_lo) : 0;
  const int n_pg = any_rows ? page_index(start + r_hi - 1) - pg0 + 1 : 0;
  const bool cached = !RT && n_pg <= kLagPtCache;
  float* red = lds + (LAG ? lagkv_range_floats(a.H, a.d, BIG) : 0);
  int* lpt = reinterpret_cast<int*>(red + (WIDE ? WAVES * AH * kRedRowWords : 0));
  if (cached)
    for (int i = tid; i < n_pg; i += NT) lpt[i] = pt[pg0 + i];
  // (RT: the same LDS holds the share's row offsets, filled below)
  int64_t* lrows = reinterpret_cast<int64_t*>(lpt);
  // The plane's base and this lane's column: a row address is the base
  // plus a wave-uniform row offset (row segments), to which the lane's
  // column is added by the load itself.
  const char* pbase = a.base + (int64_t)layer * a.s_layer + (int64_t)kv * a.s_kv;
  const int loff = col * 4 * NW;
  // Byte offset (in the plane) of chunk row r, -1 if the row is past `hi`
  // or its page is out of range.
  auto row_off = [&](int r, int hi) -> int64_t {
    if (!seq_ok || r >= hi) return -1;
    const int pos = start + r;
    const int pidx = page_index(pos);
    // (an LDS-typed read: a generic load of either table would make the
    // compiler wait for every row load in flight)
    const int pg = cached ? ((const lds_int*)lpt)[pidx - pg0] : pt[pidx];
    if (pg < 0 || pg >= a.n_pages) return -1;
    return (int64_t)pg * a.s_page + (int64_t)(pos - pidx * a.page_size) * row_bytes;
  };
  // Row segments: a wavefront walks its rows in blocks of 64; lane i
  // keeps the offset of row tb + i of the current block, and a row's
  // offset is read from it with readlane -- no memory round trip per row.
  // The table is filled at the head of each block only, so the page-table
  // arithmetic is not live in the loop over the block's rows.
  if (RT)
    for (int i = tid; i < r_hi - r_lo; i += NT) lrows[i] = row_off(r_lo + i, r_hi);
  __syncthreads();
  int tb = 0;
  uint32_t t_lo = 0, t_hi = 0;
  auto fill_table = [&](int it0) {
    if (!WIDE) return;
    tb = s_lo + it0;
    const int r = tb + lane;
    const int64_t o = RT ? (r < s_hi ? ((const lds_i64*)lrows)[r - r_lo] : -1) : row_off(r, s_hi);
    t_lo = (uint32_t)o;
    t_hi = (uint32_t)((uint64_t)o >> 32);
  };
  // (rows past the block are absent: they are loaded in the next block)
  auto row_addr = [&](int r, bool& ok) -> const char* {
    int64_t off;
    if (WIDE) {
      const int i = r - tb;
      const int ic = i < 64 ? i : 63;
      const uint32_t lo = __builtin_amdgcn_readlane(t_lo, ic);
      const uint32_t hi = __builtin_amdgcn_readlane(t_hi, ic);
      off = i < 64 ? (int64_t)(((uint64_t)hi << 32) | lo) : -1;
    } else {
      off = row_off(r, s_hi);
    }
    ok = off >= 0;
    return ok ? pbase + off : pbase;
  };
  // Row r's words for this lane; every load is issued, also past the
  // wavefront's rows (row segments: a missing row's loads are empty and
  // read 0; narrow rows: it reads the plane's first row and is ignored),
  // so that the loads in flight are the same on every path: the compiler
  // then waits for each row alone, not for the rows in flight behind it.
  auto load_row = [&](int r, uint32_t (&w)[NW], bool& ok) {
    const char* q = row_addr(r, ok);
    if (WIDE)
      ld_row_nt<NW>(q, (uint32_t)loff, ok ? row_bytes : 0, w);
    else
      ld_lane_nt<NW>(q + loff, w);
  };

  float cmn[NCH], cmx[NCH];  // this lane's channels' range over its rows
#pragma unroll
  for (int e = 0; e < NCH; ++e) {
    cmn[e] = __builtin_huge_valf();
    cmx[e] = -__builtin_huge_valf();
  }
  // The chunk's range over the workgroup's rows: every row slot (and,
  // narrow rows, row of a wavefront) leaves its partial range in its own
  // LDS slot of [2][H*d] floats (minima, then maxima); after a barrier
  // thread t reduces channels t, t + NT, ... over the slots in slot order
  // and writes the result to `dst` (the state, or this share's part for
  // the second kernel) and, with `keep`, back into slot 0.
  const int n_part = slots * rpw;
  const int vid = slot * rpw + rw;
  auto deposit = [&]() {
    float* sl = lds + (int64_t)vid * 2 * HD + col * NCH;
#pragma unroll
    for (int e = 0; e < NCH; e += 4) {
      *reinterpret_cast<float4*>(sl + e) = make_float4(cmn[e], cmn[e + 1], cmn[e + 2], cmn[e + 3]);
      *reinterpret_cast<float4*>(sl + HD + e) =
          make_float4(cmx[e], cmx[e + 1], cmx[e + 2], cmx[e + 3]);
    }
  };
  const int64_t plane_off = (((int64_t)b * a.L + layer) * 2 + kv) * HD;
  auto combine = [&](bool keep) {
    __syncthreads();
    float* dst = a.splits == 1 ? a.range_out : a.prange + (int64_t)sp * 2 * half;
    // four channels per thread and step (each half holds whole groups of 4)
    for (int i = 4 * tid; i < 2 * HD; i += 4 * NT) {
      const bool lo = i < HD;
      float4 v = *reinterpret_cast<const float4*>(lds + i);
      for (int k = 1; k < n_part; ++k) {
        const float4 o = *reinterpret_cast<const float4*>(lds + (int64_t)k * 2 * HD + i);
        v.x = lo ? nan_min(v.x, o.x) : nan_max(v.x, o.x);
        v.y = lo ? nan_min(v.y, o.y) : nan_max(v.y, o.y);
        v.z = lo ? nan_min(v.z, o.z) : nan_max(v.z, o.z);
        v.w = lo ? nan_min(v.w, o.w) : nan_max(v.w, o.w);
      }
      const int64_t at = (lo ? 0 : half - HD) + plane_off + i;
      *reinterpret_cast<float4*>(dst + at) = v;
      if (keep) *reinterpret_cast<float4*>(lds + i) = v;
      if (a.splits == 1 && !a.two) {
        // a one-tensor signal carries no range for the other tensor
        *reinterpret_cast<float4*>(a.range_out + at + (int64_t)(1 - 2 * kv) * HD) =
            make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    __syncthreads();
  };

  // y = (x - mn) * sc - 1/2: the normalisation (shifted by -1/2) of each
  // channel.  The difference comes first: folding mn * sc into the
  // addend would round at the magnitude of x * sc, which a narrow range
  // (sc up to 1/eps) makes large.
  float mnv[LAG ? NCH : 1], sc[LAG ? NCH : 1];
  if (LAG) {
    if (fresh) {
      // first pass: the chunk's own range
      for (int it = 0; it < sweeps; ++it) {
        if (it % 64 == 0) fill_table(it);
        uint32_t w[NW];
        bool ok;
        load_row(row_of(it), w, ok);
        if (ok)
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            cmn[2 * k] = nan_min(cmn[2 * k], bf16_lo(w[k]));
            cmx[2 * k] = nan_max(cmx[2 * k], bf16_lo(w[k]));
            cmn[2 * k + 1] = nan_min(cmn[2 * k + 1], bf16_hi(w[k]));
            cmx[2 * k + 1] = nan_max(cmx[2 * k + 1], bf16_hi(w[k]));
          }
      }
      deposit();
      combine(true);
    }
#pragma unroll
    for (int e = 0; e < NCH; ++e) {
      const float mn = fresh ? lds[col * NCH + e] : rin[e];
      const float mx = fresh ? lds[HD + col * NCH + e] : rin[NCH + e];
      mnv[e] = mn;
      sc[e] = __builtin_amdgcn_rcpf(mx - mn + a.eps);  // (one reciprocal instruction)
    }
  }

  const float inv_d = 1.0f / (float)a.d;
  const bf16x2 one2 = __builtin_bit_cast(bf16x2, 0x3F803F80u);  // (1, 1)
  // Variance of a head from the sum and the sum of squares of its values
  // (lag-normalised: y = (x - mn) * sc - 1/2 per channel, the variance
  // being that of x~).  A missing row is computed like any other and its
  // result dropped at the write: a load whose value might go unused forces
  // a wait for every load in flight before its register is reused.
  auto head_var = [&](float s, float q) -> float {
    const float mu = s * inv_d;
    return fmaf(-mu, mu, q * inv_d);
  };
  // raw: x0 + x1 and x0^2 + x1^2 of each packed pair in one instruction
  auto sums_raw = [&](const uint32_t (&w)[NW], float& s, float& q) {
    s = 0.f;
    q = 0.f;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const bf16x2 x = __builtin_bit_cast(bf16x2, w[k]);
      s = __builtin_amdgcn_fdot2_f32_bf16(x, one2, s, false);
      q = __builtin_amdgcn_fdot2_f32_bf16(x, x, q, false);
    }
  };

  // Transposed reduction of a batch of AH rows (row segments): lane l
  // takes the (row, head) pair l / lpp of the batch -- lpp lanes per pair
  // when a head spans more lanes than the batch has rows -- adds m =
  // gw / lpp lanes' partials in lane order, the pair's lanes combine
  // theirs, and the heads of a row (rg adjacent lanes) are summed.
  const int hs = 64 / gw;                       // heads per row segment
  const int lpp = gw > AH ? gw / AH : 1;
  const int m = gw / lpp;
  const int ppp = 64 / lpp;                     // pairs per pass
  const int passes = WIDE ? AH * hs / ppp : 0;
  const int rg = hs * lpp;
  float* red_w = red + wave * AH * kRedRowWords;
  auto put = [&](int u, float s, float q) {
    *reinterpret_cast<float2*>(red_w + u * kRedRowWords + red_word(lane)) = make_float2(s, q);
  };
  auto reduce_batch = [&](int it0, uint32_t okm) {
    wave_sync();
    for (int ps = 0; ps < passes; ++ps) {
      const int P = ps * ppp + lane / lpp;
      const int j = lane & (lpp - 1);
      const int u = P / hs;
      const int h = P - u * hs;
      const float* src = red_w + u * kRedRowWords;
      const int l0 = h * gw + j * m;
      float S = 0.f, Q = 0.f;
#pragma unroll
      for (int i = 0; i < AH; ++i)
        if (i < m) {
          const float2 v = *reinterpret_cast<const float2*>(src + red_word(l0 + i));
          S += v.x;
          Q += v.y;
        }
      S = group_sum(S, lpp);
      Q = group_sum(Q, lpp);
      const float rs = group_sum(j == 0 ? head_var(S, Q) : 0.f, rg);
      const int r = s_lo + it0 + u;
      if ((lane & (rg - 1)) == 0 && r < s_hi) part[r] = (okm >> u) & 1 ? rs : 0.f;
    }
    wave_sync();
  };

  const bool track_range = LAG && !fresh;
  // Rows u and u + 1 of the batch at sweep it0: the range, then each
  // lane's sum and sum of squares (row segments: into LDS for the batch's
  // transposed reduction; narrow rows: each head's variance, the row's
  // heads added with lane shuffles in lane order and written by the row's
  // first lane).  Rows past the share are not written.
  auto process_pair = [&](int it0, int u, const uint32_t (&wa)[NW], const uint32_t (&wb)[NW],
                          bool oka, bool okb) {
    float sa = 0.f, qa = 0.f, sb = 0.f, qb = 0.f;
    if (LAG) {
      // one packed word at a time: each value unpacked once, for the
      // range and the sums
      auto sums = [&](float xa, float xb, int e) {
        const float ya = fmaf(xa - mnv[e], sc[e], -0.5f);
        const float yb = fmaf(xb - mnv[e], sc[e], -0.5f);
        if (e == 0) {  // (the sums start at the first channel, not at 0 + y)
          sa = ya;
          qa = ya * ya;
          sb = yb;
          qb = yb * yb;
        } else {
          sa += ya;
          qa = fmaf(ya, ya, qa);
          sb += yb;
          qb = fmaf(yb, yb, qb);
        }
      };
      if (track_range && oka && okb) {
        // both rows present: three-input minimum / maximum
#pragma unroll
        for (int k = 0; k < NW; ++k) {
          const int e = 2 * k;
          const float a0 = bf16_lo(wa[k]), a1 = bf16_hi(wa[k]);
          const float b0 = bf16_lo(wb[k]), b1 = bf16_hi(wb[k]);
          cmn[e] = nan_min(cmn[e], nan_min(a0, b0));
          cmx[e] = nan_max(cmx[e], nan_max(a0, b0));
          cmn[e + 1] = nan_min(cmn[e + 1], nan_min(a1, b1));
          cmx[e + 1] = nan_max(cmx[e + 1], nan_max(a1, b1));
          sums(a0, b0, e);
          sums(a1, b1, e + 1);
        }
      } else {
#pragma unroll
        for (int k = 0; k < NW; ++k) {
          const int e = 2 * k;
          const float a0 = bf16_lo(wa[k]), a1 = bf16_hi(wa[k]);
          const float b0 = bf16_lo(wb[k]), b1 = bf16_hi(wb[k]);
          if (track_range && oka) {
            cmn[e] = nan_min(cmn[e], a0);
            cmx[e] = nan_max(cmx[e], a0);
            cmn[e + 1] = nan_min(cmn[e + 1], a1);
            cmx[e + 1] = nan_max(cmx[e + 1], a1);
          }
          if (track_range && okb) {
            cmn[e] = nan_min(cmn[e], b0);
            cmx[e] = nan_max(cmx[e], b0);
            cmn[e + 1] = nan_min(cmn[e + 1], b1);
            cmx[e + 1] = nan_max(cmx[e + 1], b1);
          }
          sums(a0, b0, e);
          sums(a1, b1, e + 1);
        }
      }
    } else {
      sums_raw(wa, sa, qa);
      sums_raw(wb, sb, qb);
    }
    if (WIDE) {
      put(u, sa, qa);
      put(u + 1, sb, qb);
      return;
    }
    float va = head_var(group_sum(sa, gw), group_sum(qa, gw));
    float vb = head_var(group_sum(sb, gw), group_sum(qb, gw));
    for (int off = gw; off < lpr; off <<= 1) {
      va += __shfl_xor(va, off, 64);
      vb += __shfl_xor(vb, off, 64);
    }
    const int r = row_of(it0 + u);
    if (li == 0 && r < s_hi) part[r] = oka ? va : 0.f;
    if (li == 0 && r + rpw < s_hi) part[r + rpw] = okb ? vb : 0.f;
  };
  // Rolling pipeline over AH rows in flight: as soon as a pair of rows is
  // used its registers receive the pair AH rows on.  Every load is
  // unconditional, so the loads in flight are the same on every path and
  // each use waits for its own pair only.
  // (in blocks of 64 sweeps: a block's last loads reach past it and are
  // empty; the next block starts its own)
  for (int b0 = 0; b0 < sweeps; b0 += 64) {
    fill_table(b0);
    const int b1 = min(sweeps, b0 + 64);
    // (okn: one bit per row in flight, set when the row is present)
    uint32_t raw[AH][NW];
    uint32_t okn = 0;
    auto load_bit = [&](int r, int u) {
      bool ok;
      load_row(r, raw[u], ok);
      okn = (okn & ~(1u << u)) | (ok ? 1u << u : 0u);
    };
#pragma unroll
    for (int u = 0; u < AH; ++u) load_bit(row_of(b0 + u), u);
    for (int it0 = b0;; it0 += AH) {
      const uint32_t okm = okn;
#pragma unroll
      for (int u = 0; u < AH; u += 2) {
        process_pair(it0, u, raw[u], raw[u + 1], (okm >> u) & 1, (okm >> (u + 1)) & 1);
        load_bit(row_of(it0 + AH + u), u);
        load_bit(row_of(it0 + AH + u + 1), u + 1);
      }
      if (WIDE) reduce_batch(it0, okm);
      if (it0 + AH >= b1) break;
    }
  }

  if (LAG && !fresh) {
    deposit();
    combine(false);
  }
}

// Blocks [0, tok_blocks) of each sequence: q(t) = the sum of token t's
// partial sums over the used planes and row segments, times 1/(L*H).  A
// block takes kRedTok tokens; its kScoreThreads / kRedTok parts each add
// every parts-th partial in order, then the parts are added in order.  The
// remaining blocks (split rows of a lag-normalised signal): each channel's
// range over the chunk = the min and max of the shares' partial ranges, in
// a fixed order.
constexpr int kRedTok = 64;
constexpr int kRedParts = kScoreThreads / kRedTok;

__global__ __launch_bounds__(kScoreThreads) void k_lag_reduce(LagReduceArgs a) {
  __shared__ float red[kRedParts][kRedTok];
  const int b = blockIdx.y;
  const int tok_blocks = (a.C + kRedTok - 1) / kRedTok;
  if ((int)blockIdx.x < tok_blocks) {
    const int t = threadIdx.x % kRedTok;
    const int part = threadIdx.x / kRedTok;
    const int c = blockIdx.x * kRedTok + t;
    float s = 0.f;
    if (c < a.C) {
      const float* p = a.partial + (int64_t)b * a.n_sums * a.C + c;
#pragma unroll 8
      for (int pl = part; pl < a.n_sums; pl += kRedParts) s += p[(int64_t)pl * a.C];
    }
    red[part][t] = s;
    __syncthreads();
    if (part == 0 && c < a.C) {
      float q = red[0][t];
#pragma unroll
      for (int k = 1; k < kRedParts; ++k) q += red[k][t];
      a.sig[(int64_t)b * a.C + c] = q * a.inv_count;
    }
    return;
  }
  const int i = ((int)blockIdx.x - tok_blocks) * kScoreThreads + threadIdx.x;
  if (i >= a.n_chan) return;
  const int64_t half = (int64_t)a.B * a.n_chan;
  const int64_t o = (int64_t)b * a.n_chan + i;
  const int kv = (i / (a.n_chan / (2 * a.L))) & 1;
  float lo = 0.f, hi = 0.f;  // planes of an unused tensor carry no range
  if (kv == 0 ? a.use_k : a.use_v) {
    lo = a.prange[o];
    hi = a.prange[half + o];
    for (int sp = 1; sp < a.splits; ++sp) {
      lo = nan_min(lo, a.prange[sp * 2 * half + o]);
      hi = nan_max(hi, a.prange[sp * 2 * half + half + o]);
    }
  }
  a.range_out[o] = lo;
  a.range_out[half + o] = hi;
}

template <bool LAG, bool WIDE, int NW, bool RT = false, bool BIG = false>
hipError_t launch_lag(const ScoreLagArgs& a, hipStream_t s) {
  const dim3 grid(a.n_planes, a.B, a.splits);
  const size_t lds = lagkv_lds_bytes(a.H, a.d, a.lag, BIG);
  hipLaunchKernelGGL((k_score_lagkv<LAG, WIDE, NW, RT, BIG>), grid, dim3(lagkv_threads(LAG, BIG)),
                     lds, s, a);
  return hipGetLastError();
}

}  // namespace

size_t lagkv_lds_bytes(int H, int d, bool lag, bool big) {
  return (lag ? lagkv_range_floats(H, d, big) * sizeof(float) : 0) +
         (lagkv_wide(H, d, lag)
              ? (size_t)lagkv_waves(lag, big) * lagkv_ahead(lag) * kRedRowWords * sizeof(float)
              : 0) +
         kLagPtCache * sizeof(int);
}

hipError_t launch_score_lagkv(const ScoreLagArgs& a, const LagReduceArgs& r, hipStream_t s) {
  const bool wide = lagkv_wide(a.H, a.d, a.lag);
  // (a stream's first chunk is one share of all C rows, so C bounds a share)
  const bool rt = a.C <= kLagRowCache;
  const bool big = lagkv_big(a.H, a.d, a.lag, (int64_t)a.n_planes * a.B);
  const hipError_t e =
      a.lag ? (!wide ? launch_lag<true, false, kLagWords>(a, s)
               : rt  ? (big ? launch_lag<true, true, kLagWords, true, true>(a, s)
                            : launch_lag<true, true, kLagWords, true>(a, s))
                     : (big ? launch_lag<true, true, kLagWords, false, true>(a, s)
                            : launch_lag<true, true, kLagWords>(a, s)))
            : (!wide ? launch_lag<false, false, kLagWords>(a, s)
               : rt  ? launch_lag<false, true, kLagWords, true>(a, s)
                     : launch_lag<false, true, kLagWords>(a, s));
  if (e != hipSuccess) return e;
  const int tok_blocks = (r.C + kRedTok - 1) / kRedTok;
  const int rng_blocks = r.lag && r.splits > 1 ? (r.n_chan + kScoreThreads - 1) / kScoreThreads : 0;
  hipLaunchKernelGGL(k_lag_reduce, dim3(tok_blocks + rng_blocks, r.B), dim3(kScoreThreads), 0, s,
                     r);
  return hipGetLastError();
}

}  // namespace epikv
