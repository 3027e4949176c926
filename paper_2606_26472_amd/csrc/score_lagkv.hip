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
// Kernel 1: one 512-thread workgroup per (sequence, used plane) -- a plane is
// one (layer, K|V) of a used tensor, so signals of one tensor launch half as
// many -- streaming the chunk's rows of that plane from the paged pool.  When
// that gives too few workgroups to fill the GPU the rows are split between
// `splits` workgroups, whose partial channel ranges the second kernel
// combines; otherwise the workgroup writes the chunk's range itself.
// A lane owns one 16-byte column = 8 channels of one head, so a head's
// statistics reduce over d/8 lanes with DPP row operations.  A wavefront
// takes a segment of 512 channels of a row (rows of 1024 channels: two
// wavefronts per row, each writing its own partial sum), or several narrow
// rows.  Each wavefront loads kLagAhead rows (page-table entries first, then
// the rows) before it uses any; with row segments the row, its page and its
// address are wave-uniform (scalar).
//   Variance, one pass: the sum and the sum of squares over the head.  For
//   the lag-normalised signals each channel is mapped to
//   y = (x - mn) / (mx - mn + eps) - 1/2 (the shift keeps the sums of
//   squares free of cancellation; a variance does not change under a
//   shift); for the raw signals the packed bf16 words feed
//   v_dot2_f32_bf16 directly (x0 + x1 and x0^2 + x1^2 in one instruction
//   each, no unpacking).
//   Range (lag-normalised, not the first chunk): IEEE minimum / maximum
//   over the rows -- a NaN propagates, as in a plain minimum over the chunk
//   -- with three-input instructions over pairs of rows; the wavefronts'
//   ranges are combined through LDS in a fixed tree.
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

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of `width` lanes (2..32); every lane of a group
// ends with the same bits (each step adds two values that the partner lane
// adds in the other order).  Within a row of 16 lanes: DPP moves (quad
// permutes, half-row mirror, rotations); across rows: a lane shuffle.
__device__ __forceinline__ float group_sum(float v, int width) {
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
  if (width == 32) v += __shfl_xor(v, 16, 64);
  return v;
}

// One 16-byte column of a row whose address is wave-uniform: a buffer
// resource made for the row (scalar registers) and the lane's byte offset
// as the only vector operand, so a row costs no vector address arithmetic.
// The resource spans the row alone (offsets past it would read 0).
// Non-temporal: each byte is read once.
__device__ __forceinline__ u32x4 ld_row_nt(const char* row, uint32_t off, int row_bytes) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)row, (short)0, row_bytes, kBufferRsrcWord3);
  return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kBufferNonTemporal);
}

__device__ __forceinline__ float nan_min(float a, float b) {
  return __builtin_elementwise_minimum(a, b);
}
__device__ __forceinline__ float nan_max(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}

// LAG: lag-normalised signal.  WIDE: rows of at least 512 channels, split
// into segments of 64 lanes x CPL 16-byte columns (8 * CPL channels per
// lane), one segment per wavefront, so the row, its page and its address
// are wave-uniform; narrower rows are shared by the lanes of one
// wavefront, 64 / row_vec rows at a time (CPL = 1).  The raw signals take
// two columns per lane for rows of 1024 channels or more, which halves the
// per-row work (cross-lane sums, addressing) per channel; the
// lag-normalised form keeps one (its per-channel range and normalisation
// would not fit 128 registers with two).
template <bool LAG, bool WIDE, int CPL>
__global__ __launch_bounds__(kLagThreads) __attribute__((amdgpu_waves_per_eu(4)))
void k_score_lagkv(ScoreLagArgs a) {
  constexpr int NCH = 8 * CPL;  // channels per lane
  constexpr int AH = kLagAhead;  // rows per batch
  static_assert(!(LAG && CPL > 1), "the lag-normalised form takes one column per lane");
  extern __shared__ float lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int p = blockIdx.x;     // used plane
  const int b = blockIdx.y;
  const int sp = blockIdx.z;    // share of the chunk's rows
  const int layer = a.two ? p >> 1 : p;
  const int kv = a.two ? (p & 1) : a.kv0;
  const int HD = a.H * a.d;
  const int row_vec = HD >> 3;                    // 16-byte columns per row
  const int segs = WIDE ? row_vec / (64 * CPL) : 1;  // wavefronts per row
  const int lpr = WIDE ? 64 : row_vec;            // lanes per row segment
  const int rpw = WIDE ? 1 : 64 / row_vec;        // rows per wavefront
  const int seg = WIDE ? wave % segs : 0;         // this wavefront's segment
  const int slot = WIDE ? wave / segs : wave;     // its row slot in the workgroup
  const int rw = WIDE ? 0 : lane / lpr;           // this lane's row within the wavefront's
  const int li = lane - rw * lpr;                 // lane within the segment
  const int col = seg * 64 + li;                  // this lane's group of CPL columns
  const int gw = a.d / NCH;                       // lanes per head
  const int row_bytes = HD * 2;

  const int N = a.n_cached[b];
  const int start = N - a.C;
  const bool seq_ok = start >= 0 && (int64_t)((N - 1) / a.page_size) < a.ld_pt;
  const int32_t* pt = a.pt + (int64_t)b * a.ld_pt;
  const int64_t half = (int64_t)a.B * a.L * 2 * HD;
  // this lane's first channel in the [2][B][L][2][H][d] range layout
  const int64_t rbase = (((int64_t)b * a.L + layer) * 2 + kv) * HD + col * NCH;
  const bool fresh = LAG && a.n_tok_in[b] <= 0;
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
  const int slots = kLagWaves / segs;                     // row slots of the workgroup
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
  const bool cached = n_pg <= kLagPtCache;
  int* lpt = reinterpret_cast<int*>(lds + (LAG ? lagkv_tree_floats(a.H, a.d) : 0));
  if (cached)
    for (int i = tid; i < n_pg; i += kLagThreads) lpt[i] = pt[pg0 + i];
  __syncthreads();
  // The plane's base and this lane's column: a row address is the base
  // plus a wave-uniform row offset (row segments), to which the lane's
  // column is added by the load itself.
  const char* pbase = a.base + (int64_t)layer * a.s_layer + (int64_t)kv * a.s_kv;
  const int loff = col * 16 * CPL;
  // Byte offset (in the plane) of chunk row r, -1 if the row is not this
  // wavefront's or its page is out of range.
  auto row_off = [&](int r) -> int64_t {
    if (!seq_ok || r >= s_hi) return -1;
    const int pos = start + r;
    const int pidx = page_index(pos);
    const int pg = cached ? lpt[pidx - pg0] : pt[pidx];
    if (pg < 0 || pg >= a.n_pages) return -1;
    return (int64_t)pg * a.s_page + (int64_t)(pos - pidx * a.page_size) * row_bytes;
  };
  // Row segments: lane i keeps the offset of row tb + i of the wavefront's
  // block (a table refilled every 64 rows), and a row's offset is read
  // from it with readlane -- no memory round trip per row, and (the table
  // being computed, not loaded) no wait for the rows in flight.
  int tb = -(1 << 30);
  uint32_t t_lo = 0, t_hi = 0;
  auto row_addr = [&](int r, bool& ok) -> const char* {
    int64_t off;
    if (WIDE) {
      if (r - tb >= 64 || r < tb) {
        tb = r;
        const int64_t o = row_off(r + lane);
        t_lo = (uint32_t)o;
        t_hi = (uint32_t)((uint64_t)o >> 32);
      }
      const uint32_t lo = __builtin_amdgcn_readlane(t_lo, r - tb);
      const uint32_t hi = __builtin_amdgcn_readlane(t_hi, r - tb);
      off = (int64_t)(((uint64_t)hi << 32) | lo);
    } else {
      off = row_off(r);
    }
    ok = off >= 0;
    return ok ? pbase + off : pbase;
  };
  // Load the rows of sweeps it0 .. it0 + kLagAhead - 1; ok[u]: row present.
  // Every load is issued (a missing row reads the plane's first row and is
  // ignored), so the loads are straight-line code and the compiler can
  // wait for each batch alone rather than for every load in flight.
  auto load_rows = [&](int it0, u32x4 (&raw)[AH][CPL], bool (&ok)[AH]) {
#pragma unroll
    for (int u = 0; u < AH; ++u) {
      const char* q = row_addr(row_of(it0 + u), ok[u]);
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        raw[u][c] = WIDE ? ld_row_nt(q, (uint32_t)(loff + 16 * c), row_bytes)
                         : ld_stream(q + loff + 16 * c);
    }
  };

  float cmn[NCH], cmx[NCH];  // this lane's channels' range over its rows
#pragma unroll
  for (int e = 0; e < NCH; ++e) {
    cmn[e] = __builtin_huge_valf();
    cmx[e] = -__builtin_huge_valf();
  }
  auto unpack = [](const u32x4 (&w)[CPL], float (&x)[NCH]) {
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        x[c * 8 + 2 * k] = bf16_lo(w[c][k]);
        x[c * 8 + 2 * k + 1] = bf16_hi(w[c][k]);
      }
  };
  auto track = [&](const float (&x)[NCH]) {
#pragma unroll
    for (int e = 0; e < NCH; ++e) {
      cmn[e] = nan_min(cmn[e], x[e]);
      cmx[e] = nan_max(cmx[e], x[e]);
    }
  };
  // Combine the range over the workgroup's row slots (and the rows of one
  // wavefront) in a fixed tree through LDS, slots of [2][H*d] floats; the
  // partial of slot 0 ends with the result.  With `bcast` every lane then
  // reads it.
  const int n_part = slots * rpw;
  const int vid = slot * rpw + rw;
  auto combine = [&](bool bcast) {
    for (int s = n_part / 2; s >= 1; s >>= 1) {
      if (vid >= s && vid < 2 * s) {
        float* sl = lds + (int64_t)(vid - s) * 2 * HD + col * NCH;
#pragma unroll
        for (int e = 0; e < NCH; ++e) {
          sl[e] = cmn[e];
          sl[HD + e] = cmx[e];
        }
      }
      __syncthreads();
      if (vid < s) {
        const float* sl = lds + (int64_t)vid * 2 * HD + col * NCH;
#pragma unroll
        for (int e = 0; e < NCH; ++e) {
          cmn[e] = nan_min(cmn[e], sl[e]);
          cmx[e] = nan_max(cmx[e], sl[HD + e]);
        }
      }
      __syncthreads();
    }
    if (bcast) {
      if (vid == 0) {
#pragma unroll
        for (int e = 0; e < NCH; ++e) {
          lds[col * NCH + e] = cmn[e];
          lds[HD + col * NCH + e] = cmx[e];
        }
      }
      __syncthreads();
#pragma unroll
      for (int e = 0; e < NCH; ++e) {
        cmn[e] = lds[col * NCH + e];
        cmx[e] = lds[HD + col * NCH + e];
      }
    }
  };

  // y = (x - mn) * sc - 1/2: the normalisation (shifted by -1/2) of each
  // channel.  The difference comes first: folding mn * sc into the
  // addend would round at the magnitude of x * sc, which a narrow range
  // (sc up to 1/eps) makes large.
  float mnv[LAG ? NCH : 1], sc[LAG ? NCH : 1];
  if (LAG) {
    if (fresh) {
      // first pass: the chunk's own range
      for (int it0 = 0; it0 < sweeps; it0 += AH) {
        u32x4 raw[AH][CPL];
        bool ok[AH];
        load_rows(it0, raw, ok);
#pragma unroll
        for (int u = 0; u < AH; ++u) {
          float x[NCH];
          unpack(raw[u], x);
          if (ok[u]) track(x);
        }
      }
      combine(true);
    }
#pragma unroll
    for (int e = 0; e < NCH; ++e) {
      const float mn = fresh ? cmn[e] : a.range_in[rbase + e];
      const float mx = fresh ? cmx[e] : a.range_in[half + rbase + e];
      mnv[e] = mn;
      sc[e] = 1.0f / (mx - mn + a.eps);
    }
  }

  const float inv_d = 1.0f / (float)a.d;
  const bf16x2 one2 = __builtin_bit_cast(bf16x2, 0x3F803F80u);  // (1, 1)
  // Variance of this lane's head for one row from the sum and the sum of
  // squares of its values (lag-normalised: y = (x - mn) * sc - 1/2 per
  // channel, the variance being that of x~): every lane of the wavefront runs it (the group sums see every
  // lane of a group).  A missing row is computed like any other and its
  // result dropped at the write: a load whose value might go unused forces
  // a wait for every load in flight before its register is reused.
  auto finish_var = [&](float s, float q) -> float {
    s = group_sum(s, gw);
    q = group_sum(q, gw);
    const float mu = s * inv_d;
    return fmaf(-mu, mu, q * inv_d);
  };
  // raw: x0 + x1 and x0^2 + x1^2 of each packed pair in one instruction
  auto var_raw = [&](const u32x4 (&w)[CPL]) -> float {
    float s = 0.f, q = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        // (through a scalar: a bit cast of the vector element itself
        // reads element 0)
        const uint32_t wk = w[c][k];
        const bf16x2 x = __builtin_bit_cast(bf16x2, wk);
        s = __builtin_amdgcn_fdot2_f32_bf16(x, one2, s, false);
        q = __builtin_amdgcn_fdot2_f32_bf16(x, x, q, false);
      }
    return finish_var(s, q);
  };

  const bool track_range = LAG && !fresh;
  // Rows of sweeps it0 .. it0 + kLagAhead - 1: the range, then each head's
  // variance, written by the head's first lane (rows past the share are
  // not written).
  auto process = [&](int it0, const u32x4 (&raw)[AH][CPL], const bool (&ok)[AH]) {
    float v[AH];
    if (LAG) {
      // rows in pairs, one packed word at a time: each value unpacked
      // once, for the range and the sums
#pragma unroll
      for (int u = 0; u < AH; u += 2) {
        float sa = 0.f, qa = 0.f, sb = 0.f, qb = 0.f;
        auto sums = [&](float xa, float xb, int e) {
          const float ya = fmaf(xa - mnv[e], sc[e], -0.5f);
          const float yb = fmaf(xb - mnv[e], sc[e], -0.5f);
          sa += ya;
          qa = fmaf(ya, ya, qa);
          sb += yb;
          qb = fmaf(yb, yb, qb);
        };
        if (track_range && WIDE && ok[u] && ok[u + 1]) {
#pragma unroll
          for (int c = 0; c < CPL; ++c)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int e = c * 8 + 2 * k;
              const float a0 = bf16_lo(raw[u][c][k]), a1 = bf16_hi(raw[u][c][k]);
              const float b0 = bf16_lo(raw[u + 1][c][k]), b1 = bf16_hi(raw[u + 1][c][k]);
              cmn[e] = nan_min(cmn[e], nan_min(a0, b0));
              cmx[e] = nan_max(cmx[e], nan_max(a0, b0));
              cmn[e + 1] = nan_min(cmn[e + 1], nan_min(a1, b1));
              cmx[e + 1] = nan_max(cmx[e + 1], nan_max(a1, b1));
              sums(a0, b0, e);
              sums(a1, b1, e + 1);
            }
        } else {
#pragma unroll
          for (int c = 0; c < CPL; ++c)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int e = c * 8 + 2 * k;
              const float a0 = bf16_lo(raw[u][c][k]), a1 = bf16_hi(raw[u][c][k]);
              const float b0 = bf16_lo(raw[u + 1][c][k]), b1 = bf16_hi(raw[u + 1][c][k]);
              if (track_range && ok[u]) {
                cmn[e] = nan_min(cmn[e], a0);
                cmx[e] = nan_max(cmx[e], a0);
                cmn[e + 1] = nan_min(cmn[e + 1], a1);
                cmx[e + 1] = nan_max(cmx[e + 1], a1);
              }
              if (track_range && ok[u + 1]) {
                cmn[e] = nan_min(cmn[e], b0);
                cmx[e] = nan_max(cmx[e], b0);
                cmn[e + 1] = nan_min(cmn[e + 1], b1);
                cmx[e + 1] = nan_max(cmx[e + 1], b1);
              }
              sums(a0, b0, e);
              sums(a1, b1, e + 1);
            }
        }
        v[u] = finish_var(sa, qa);
        v[u + 1] = finish_var(sb, qb);
      }
    } else {
#pragma unroll
      for (int u = 0; u < AH; ++u) v[u] = var_raw(raw[u]);
    }
#pragma unroll
    for (int u = 0; u < AH; ++u) {
      const int r = row_of(it0 + u);
      // the heads of the segment summed in lane order: with row segments
      // one lane per head group is read into a scalar, narrow rows add
      // their groups with lane shuffles
      float sum;
      if (WIDE) {
        sum = 0.f;
        for (int g = 0; g < 64; g += gw)
          sum += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[u]), g));
      } else {
        sum = v[u];
        for (int off = gw; off < lpr; off <<= 1) sum += __shfl_xor(sum, off, 64);
      }
      if (li == 0 && r < s_hi) part[r] = ok[u] ? sum : 0.f;
    }
  };
  // Software pipelined over two buffers: the next batch of rows is in
  // flight while this one is used.
  u32x4 ra[AH][CPL], rb[AH][CPL];
  bool oa[AH], ob[AH];
  if (sweeps > 0) load_rows(0, ra, oa);
  for (int it0 = 0; it0 < sweeps; it0 += 2 * AH) {
    if (it0 + AH < sweeps) load_rows(it0 + AH, rb, ob);
    process(it0, ra, oa);
    if (it0 + AH >= sweeps) break;
    if (it0 + 2 * AH < sweeps) load_rows(it0 + 2 * AH, ra, oa);
    process(it0 + AH, rb, ob);
  }

  if (LAG) {
    if (!fresh) combine(false);
    if (vid == 0) {
      // the chunk's range: straight into the state when one workgroup saw
      // every row, else this share's part for the second kernel
      float* dst = a.splits == 1 ? a.range_out : a.prange + (int64_t)sp * 2 * half;
#pragma unroll
      for (int e = 0; e < NCH; ++e) {
        dst[rbase + e] = cmn[e];
        dst[half + rbase + e] = cmx[e];
      }
      if (a.splits == 1 && !a.two) {
        // a one-tensor signal carries no range for the other tensor
        const int64_t other = rbase + (int64_t)(1 - 2 * kv) * HD;
#pragma unroll
        for (int e = 0; e < NCH; ++e) {
          a.range_out[other + e] = 0.f;
          a.range_out[half + other + e] = 0.f;
        }
      }
    }
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

template <bool WIDE, int CPL>
hipError_t launch_lag(const ScoreLagArgs& a, hipStream_t s) {
  const dim3 grid(a.n_planes, a.B, a.splits);
  const size_t lds = lagkv_lds_bytes(a.H, a.d, a.lag);
  if (CPL == 1 && a.lag)
    hipLaunchKernelGGL((k_score_lagkv<true, WIDE, 1>), grid, dim3(kLagThreads), lds, s, a);
  else
    hipLaunchKernelGGL((k_score_lagkv<false, WIDE, CPL>), grid, dim3(kLagThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace

size_t lagkv_lds_bytes(int H, int d, bool lag) {
  return (lag ? lagkv_tree_floats(H, d) * sizeof(float) : 0) + kLagPtCache * sizeof(int);
}

hipError_t launch_score_lagkv(const ScoreLagArgs& a, const LagReduceArgs& r, hipStream_t s) {
  const int cpl = lagkv_cpl(a.H, a.d, a.lag);
  const int row_vec = a.H * a.d / 8;
  const hipError_t e = cpl == 2        ? launch_lag<true, 2>(a, s)
                       : row_vec >= 64 ? launch_lag<true, 1>(a, s)
                                       : launch_lag<false, 1>(a, s);
  if (e != hipSuccess) return e;
  const int tok_blocks = (r.C + kRedTok - 1) / kRedTok;
  const int rng_blocks = r.lag && r.splits > 1 ? (r.n_chan + kScoreThreads - 1) / kScoreThreads : 0;
  hipLaunchKernelGGL(k_lag_reduce, dim3(tok_blocks + rng_blocks, r.B), dim3(kScoreThreads), 0, s,
                     r);
  return hipGetLastError();
}

}  // namespace epikv
