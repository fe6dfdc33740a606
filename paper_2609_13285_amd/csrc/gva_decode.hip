// libgva.so -- GVA decode-step attention for MI355X (gfx950, CDNA4).
//
// The method is Grouped Value Attention with decoupled RoPE: the cache keeps
// G value streams plus one shared, already-rotated positional key; the
// per-head key map M_h is absorbed into the query (eq. absorb, Section 3.2),
// so the content score against cached position t is q~_h . v_t and no
// content key is ever formed (Section 3.3, Algorithm 1).
//
// Kernels
//   append_kernel        Algorithm 1 append steps + eq. krope (fp64 rotation)
//   absorb_bf16_kernel   eq. absorb + query rotation on the matrix cores
//   absorb_f32_kernel    the same on the vector ALUs, fp32 storage
//   decode_bf16_kernel   the hot path: split-KV streaming over the value and
//                        positional-key rows of one (sequence, group, split)
//                        on the matrix cores, online softmax, optional fused
//                        absorption prologue
//   decode_f32_kernel    fp32-storage variant on the vector ALUs
//   combine_kernel       log-sum-exp merge of the split partials
//
// Cache layout (MFMA-native).  Each (sequence, group) value stream and each
// sequence's positional-key stream is stored in tiles of 16 rows; inside a
// tile the row pieces of 16 bytes are ordered piece-major:
//   element (t, i) of a stream with D columns of E bytes, P = 16/E:
//     (t/16)*16*D + ((i/P)*16 + t%16)*P + i%P
// A wave's 16-byte-per-lane load of 64 consecutive pieces then covers 1 KB
// of contiguous memory while every lane receives exactly the 8 bf16 of one
// row that its matrix-core operand slot needs (row = lane%16, columns
// 8*(lane/16) .. +7 of a 32-column chunk).
//
// Hot-loop design (bf16).  A workgroup owns one (b, g, split); its 4 waves
// take interleaved 32-row tiles and keep DEPTH tiles in registers.  Every V
// tile serves all H/G heads of the group:
//   scores  S^T[t][n] = V[t][:] . Bq[:][n]           (v_mfma 16x16x32 bf16)
//           column n holds one head's absorbed query as a bf16 high part or
//           low part (q~ = hi + lo to ~2^-16); the columns are mirrored so a
//           DPP mirror adds the pair; the positional key rides as one more
//           K-chunk of the same product
//   P.V     O^T[i][n] += V^T[i][t] P[t][n]            (v_mfma 16x16x32 bf16)
//           V^T comes from an identity-selector MFMA on the same registers;
//           P is split hi + lo again, so both products keep ~fp32 accuracy
// The score layout the MFMA returns (lane = column, registers = 4 rows) is
// exactly the B-operand layout of the P.V product, so the softmax needs no
// cross-lane traffic except the max over the four 16-lane rows.

#include <mutex>

#include "gva_common.h"

namespace {

// ================================================================ append
// One workgroup per new row.  The value pieces are loaded before seq/pos are
// known (they are indexed by the row alone), so the kernel makes a single
// dependent round trip to memory.
template <typename T>
__global__ void __launch_bounds__(256) append_kernel(AppendParams p) {
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  constexpr int P = 16 / sizeof(T);
  const int pieces_per_row = p.d_v / P;
  const int n_pieces = p.G * pieces_per_row;
  const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const T*>(p.v_new) + (int64_t)r * p.G * p.d_v);
  u32x4 piece = {0u, 0u, 0u, 0u};
  if (tid < n_pieces) piece = src[tid];
  const T* kin = static_cast<const T*>(p.kr_new) + (int64_t)r * p.d_r;
  double k0 = 0.0, k1 = 0.0;
  const bool has_pair = tid < p.d_r / 2;
  if (has_pair) {
    k0 = load_elem<T>(kin, 2 * tid);
    k1 = load_elem<T>(kin, 2 * tid + 1);
  }
  const int b = p.seq[r], ps = p.pos[r];
  if (b < 0 || b >= p.B || ps < 0 || ps >= p.t_max) return;
  // the stream holding row ps: a contiguous (b, g) stream, or, paged, the
  // page block_table[b][ps / page_rows] (rows naming a page outside the pool
  // are skipped)
  int64_t vstream0, kstream0, vstride;
  int row = ps;
  if (p.block_table != nullptr) {
    const int page = p.block_table[(int64_t)b * p.max_pages + ps / p.page_rows];
    if (page < 0 || page >= p.n_pages) return;
    row = ps % p.page_rows;
    vstride = (int64_t)p.page_rows * p.d_v;
    vstream0 = (int64_t)page * p.G * vstride;
    kstream0 = (int64_t)page * p.page_rows * p.d_r;
  } else {
    vstride = (int64_t)p.t_max * p.d_v;
    vstream0 = (int64_t)b * p.G * vstride;
    kstream0 = (int64_t)b * p.t_max * p.d_r;
  }
  for (int idx = tid; idx < n_pieces; idx += blockDim.x) {
    if (idx != tid) piece = src[idx];
    const int g = idx / pieces_per_row, c = idx % pieces_per_row;
    T* stream = static_cast<T*>(p.v_cache) + vstream0 + g * vstride;
    *reinterpret_cast<u32x4*>(stream + tiled_off<T>(row, c * P, p.d_v)) = piece;
  }
  // positional key: rotate pair i at position ps in fp64 (eq. krope)
  if (has_pair) {
    T* kstream = static_cast<T*>(p.kr_cache) + kstream0;
    double y0, y1;
    rotate_pair(k0, k1, (double)ps * p.inv_freq[tid], y0, y1);
    const int64_t o = tiled_off<T>(row, 2 * tid, p.d_r);  // the pair shares a piece
    store_from_f64<T>(kstream, o, y0);
    store_from_f64<T>(kstream, o + 1, y1);
  }
}

// ================================================================ absorb
// Position of query row r: a sequence's n_per_seq query rows are its last
// n_per_seq cached rows (one row, at L-1, for a decode step).
__device__ __forceinline__ int query_pos(const AbsorbParams& p, int r) {
  const int seq = r / p.n_per_seq, i = r % p.n_per_seq;
  const int pos = clamp_len(p.lens, seq, p.t_max) - p.n_per_seq + i;
  return pos > 0 ? pos : 0;
}

// bf16, matrix cores.  Workgroup = (head h, 16 RB query rows); wave w
// computes the output blocks ib = w, w+4, ... of
// q~^T[i][r] = sum_k M_h[i][k] q[r][h][k] (A = rows of M_h, B = the query
// rows, K = d_c).  M_h is staged through LDS in passes of 128 rows x 128
// columns: the workgroup reads each pass as whole rows (16 threads x 16 B
// per row, so every load covers whole cache lines; the MFMA operand order,
// 64 bytes of 16 rows per load, took four times as long to arrive), and the
// waves take their A operands from LDS (rows padded by 16 bytes: the 16
// rows of an operand fall in distinct banks).
constexpr int kAbsorbRows = 128, kAbsorbCols = 128, kAbsorbStride = kAbsorbCols + 8;
constexpr int kAbsorbMaxRB = 4;

__global__ void __launch_bounds__(kThreads) absorb_bf16_kernel(AbsorbParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t ms[kAbsorbRows * kAbsorbStride];
  const int h = blockIdx.x;
  const int RB = p.row_blocks;                            // M_h rows reused for RB row blocks
  const int b0 = blockIdx.y * 16 * RB;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, qd = lane >> 4;
  const int W = p.d_c + p.d_r;
  const int nck = p.d_c / 32;
  const uint16_t* qg = static_cast<const uint16_t*>(p.q);
  const uint16_t* mh = static_cast<const uint16_t*>(p.m) + (int64_t)h * p.d_v * p.d_c;
  const int nseg = (p.d_c + kAbsorbCols - 1) / kAbsorbCols;
  constexpr int kFill = kAbsorbRows * kAbsorbCols / 8 / kThreads;   // 16-byte pieces per thread and pass
  for (int rbase = 0; rbase < p.d_v; rbase += kAbsorbRows) {
    f32x4 acc[2][kAbsorbMaxRB];
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int rb = 0; rb < kAbsorbMaxRB; ++rb) acc[k2][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int seg = 0; seg < nseg; ++seg) {
      u32x4 piece[kFill];
#pragma unroll
      for (int k = 0; k < kFill; ++k) {
        const int pc = tid + kThreads * k, row = pc >> 4, col = seg * kAbsorbCols + 8 * (pc & 15);
        piece[k] = (rbase + row < p.d_v && col < p.d_c)
                       ? *reinterpret_cast<const u32x4*>(mh + (int64_t)(rbase + row) * p.d_c + col)
                       : u32x4{0u, 0u, 0u, 0u};
      }
      // the query rows' chunks of this segment, requested with the pass (one
      // memory round trip for both)
      u32x4 xq[kAbsorbMaxRB][4];
#pragma unroll
      for (int rb = 0; rb < kAbsorbMaxRB; ++rb) {
        const int bq = min(b0 + 16 * rb + n, p.B - 1);    // rows past B compute a duplicate
        const uint16_t* qrow = qg + ((int64_t)bq * p.H + h) * W + seg * kAbsorbCols + 8 * qd;
#pragma unroll
        for (int c = 0; c < 4; ++c)
          xq[rb][c] = (rb < RB && seg * 4 + c < nck) ? *reinterpret_cast<const u32x4*>(qrow + 32 * c)
                                                      : u32x4{0u, 0u, 0u, 0u};
      }
      if (rbase > 0 || seg > 0) __syncthreads();         // the previous pass has been read
#pragma unroll
      for (int k = 0; k < kFill; ++k) {
        const int pc = tid + kThreads * k;
        *reinterpret_cast<u32x4*>(ms + (pc >> 4) * kAbsorbStride + 8 * (pc & 15)) = piece[k];
      }
      __syncthreads();
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int ibl = w + kWaves * k2;                  // 16-row block of the pass
        if (rbase + 16 * ibl >= p.d_v) break;
        bf16x8 a[4];
#pragma unroll
        for (int c = 0; c < 4; ++c)
          a[c] = *reinterpret_cast<const bf16x8*>(ms + (16 * ibl + n) * kAbsorbStride + 32 * c + 8 * qd);
#pragma unroll
        for (int rb = 0; rb < kAbsorbMaxRB; ++rb) {
          if (rb >= RB || b0 + 16 * rb >= p.B) break;
#pragma unroll
          for (int c = 0; c < 4; ++c)
            if (seg * 4 + c < nck) acc[k2][rb] = mfma16(a[c], as_bf16x8(xq[rb][c]), acc[k2][rb]);
        }
      }
    }
    // lane (n, qd) holds q~[r0 + n][rbase + 16 ibl + 4 qd + jj]
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int i0 = rbase + 16 * (w + kWaves * k2);
      if (i0 >= p.d_v) break;
#pragma unroll
      for (int rb = 0; rb < kAbsorbMaxRB; ++rb) {
        const int r0 = b0 + 16 * rb;
        if (rb >= RB || r0 >= p.B) break;
        if (r0 + n < p.B)
          *reinterpret_cast<f32x4*>(p.q_abs + ((int64_t)(r0 + n) * p.H + h) * p.d_v + i0 + 4 * qd) = acc[k2][rb];
      }
    }
  }
  // the positional pairs of the workgroup's rows: 16 RB d_r / 2 tasks
  const int npair = p.d_r / 2;
  for (int task = tid; task < 16 * RB * npair; task += kThreads) {
    const int pb = b0 + task / npair, pi = task % npair;
    if (pb >= p.B) break;
    const uint32_t two = *reinterpret_cast<const uint32_t*>(qg + ((int64_t)pb * p.H + h) * W + p.d_c + 2 * pi);
    float y0, y1;
    rotate_query_pair(bf16_bits_to_f32(two & 0xFFFFu), bf16_bits_to_f32(two >> 16),
                      (double)query_pos(p, pb) * p.inv_freq[pi], 1.f, y0, y1);
    float* out = p.q_rot + ((int64_t)pb * p.H + h) * p.d_r + 2 * pi;
    out[0] = y0;
    out[1] = y1;
  }
}

// fp32 storage, vector ALUs: one workgroup per (b, h).
// sum_k x[k] y[k] over fp32 rows of n.  Rows that are 16-byte aligned with
// n a multiple of 4 are read as 16-byte pieces, eight of each row requested
// per step (32 terms per memory round trip); any others element by element,
// eight per step.
__device__ __forceinline__ float dot_f32(const float* x, const float* y, int n) {
  if ((((uintptr_t)x | (uintptr_t)y) & 15) == 0 && (n & 3) == 0) {
    const f32x4* x4 = reinterpret_cast<const f32x4*>(x);
    const f32x4* y4 = reinterpret_cast<const f32x4*>(y);
    const int n4 = n >> 2;
    f32x4 a4 = {0.f, 0.f, 0.f, 0.f};
    int k = 0;
    for (; k + 8 <= n4; k += 8) {
      f32x4 xv[8], yv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        xv[j] = x4[k + j];
        yv[j] = y4[k + j];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) a4[e] = fmaf(xv[j][e], yv[j][e], a4[e]);
    }
    for (; k < n4; ++k) {
      const f32x4 xv = x4[k], yv = y4[k];
#pragma unroll
      for (int e = 0; e < 4; ++e) a4[e] = fmaf(xv[e], yv[e], a4[e]);
    }
    return (a4[0] + a4[1]) + (a4[2] + a4[3]);
  }
  float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  int k = 0;
  for (; k + 8 <= n; k += 8) {
    float xv[8], yv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      xv[j] = x[k + j];
      yv[j] = y[k + j];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) acc8[j] = fmaf(xv[j], yv[j], acc8[j]);
  }
  for (; k < n; ++k) acc8[0] = fmaf(x[k], y[k], acc8[0]);
  return ((acc8[0] + acc8[1]) + (acc8[2] + acc8[3])) + ((acc8[4] + acc8[5]) + (acc8[6] + acc8[7]));
}

__global__ void __launch_bounds__(128) absorb_f32_kernel(AbsorbParams p) {
  const int bh = blockIdx.x;
  const int b = bh / p.H, h = bh % p.H;
  const int W = p.d_c + p.d_r;
  const float* q = static_cast<const float*>(p.q) + (int64_t)bh * W;
  const float* m = static_cast<const float*>(p.m) + (int64_t)h * p.d_v * p.d_c;
  for (int i = threadIdx.x; i < p.d_v; i += blockDim.x) {
    p.q_abs[(int64_t)bh * p.d_v + i] = dot_f32(q, m + (int64_t)i * p.d_c, p.d_c);
  }
  const int pos = query_pos(p, b);
  for (int i = threadIdx.x; i < p.d_r / 2; i += blockDim.x) {
    double y0, y1;
    rotate_pair(q[p.d_c + 2 * i], q[p.d_c + 2 * i + 1], (double)pos * p.inv_freq[i], y0, y1);
    p.q_rot[(int64_t)bh * p.d_r + 2 * i] = (float)y0;
    p.q_rot[(int64_t)bh * p.d_r + 2 * i + 1] = (float)y1;
  }
}

// ========================================================= decode (bf16)
// HPG heads per group, DV value width, NRC = ceil(d_r / 32) positional
// K-chunks, DEPTH tiles of V held in registers (DEPTH-1 loads in flight).
template <int HPG, int DV, int NRC, int NW, bool GQA>
struct DecodeCfg {
  static constexpr int NC = DV / 32;                         // K-chunks per V row
  static constexpr int NB = DV / 16;                         // 16-wide i-blocks of the output
  // (eight-wave workgroups keep three tiles in flight at d_v = 64: five
  // measured 1 us slower on the 350M shape)
  static constexpr int DEPTH = DV >= 128 ? 2 : (NW > kWaves ? 4 : 3);
  // fused absorption: 16-byte pieces of M_h per lane and load round, one
  // round of 32 where the registers allow it (no spills), else rounds of 16
  static constexpr int AR = (DV >= 128 && NRC < 2 && NW <= 8) ? 32 : 16;
  static constexpr int QS_STRIDE = DV + 4;                   // padded LDS rows (floats)
  static constexpr int QR_STRIDE = 32 * NRC + 4;
  static constexpr int LDS_PRO = HPG * (QS_STRIDE + QR_STRIDE);
  static constexpr int LDS_RED = NW * HPG * (DV + 2);
  static constexpr int LDS_FLOATS = LDS_PRO > LDS_RED ? LDS_PRO : LDS_RED;
};

// GQA = true builds the matched grouped-query baseline the paper compares
// against (Section 2): the scores read an explicit, already-rotated key
// stream per group instead of the value rows, with no positional term and
// the raw query; P.V, the softmax, the splits and the layout are shared, so
// the two kernels differ only in the bytes they must stream.
// PAGED reads the caches from page pools through a block table: only the
// addressing of a tile (and of the current row) changes.
// KR_STREAM loads the positional-key tiles with the non-temporal policy too
// (decode_kr_stream decides).
template <int HPG, int DV, int NRC, bool GQA, bool FUSED, bool PAGED, bool KR_STREAM = false, int NW = kWaves>
__global__ void __launch_bounds__(64 * NW, NW == kWaves ? 2 : 1) decode_bf16_kernel(DecodeParams p) {
  static_assert(!(GQA && FUSED), "the GQA baseline takes the raw query");
  static_assert(!(GQA && PAGED), "the GQA baseline reads contiguous caches");
  const DecodeArgs a = p.a;
  request_args<FUSED || GQA>(a);
  using Cfg = DecodeCfg<HPG, DV, NRC, NW, GQA>;
  constexpr int NT = 64 * NW;                  // threads per workgroup
  using TileT = Tile<DV, NRC, GQA>;
  constexpr int NC = Cfg::NC, NB = Cfg::NB, DEPTH = Cfg::DEPTH, AR = Cfg::AR;
  __shared__ __attribute__((aligned(16))) float lds[Cfg::LDS_FLOATS];

  int b, s, g;
  bool empty_slot;
  if (!work_item(a, b, s, g, empty_slot)) return;   // grid padding
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, uniform (SGPR)
  const int n = lane & 15, qd = lane >> 4;     // MFMA column / row slot and 16-lane row
  const int h0 = g * HPG;
  // Column roles: [hi_0 .. hi_{HPG-1}, lo_{HPG-1} .. lo_0, zero padding].
  const bool active = n < 2 * HPG;
  const bool is_lo = n >= HPG;
  const int col_head = !active ? 0 : (is_lo ? 2 * HPG - 1 - n : n);
  const int hq = h0 + col_head;
  const bf16x8 zero8 = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
  __shared__ __attribute__((aligned(16))) uint16_t prow[DV + 32 * (NRC > 0 ? NRC : 1)];
  __shared__ int32_t split_pages[PAGED ? kMaxPages : 1];   // paged: this split's page ids

  // The rows of this split are settled once the query loads are on their
  // way (they do not depend on the length), which takes a memory round trip
  // off the prologue.  The length is a scalar load through the constant
  // address space, requested here and waited for at first use.
  const int len_b = *(const __attribute__((address_space(4))) int32_t*)(a.lens + b);
  int L = 0, r0 = 0, r1 = 0;
  auto settle_rows = [&]() {
    L = len_b < 0 ? 0 : (len_b > a.t_max ? a.t_max : len_b);
    split_rows(L, a.S, a.split_rows, s, r0, r1);
    return r0 < r1 || s == 0;
  };
  auto write_empty = [&]() {                   // an empty split past the first: lse only
    if (tid < HPG) a.lse_part[((int64_t)b * a.H + h0 + tid) * a.S + s] = -INFINITY;
  };
  if (empty_slot && s > 0) {                   // bounded chunks: a split with no rows
    write_empty();
    return;
  }

  // ---- loads that do not depend on the length, oldest first: the current
  // token's rows (staged first, below), then the query.  Loads retire in
  // order, so waiting for them never waits for the tiles requested later.
  // (kept as loaded bits: converting them here would wait for them here)
  u32x4 pend_piece = {0u, 0u, 0u, 0u};
  uint32_t pend_kbits = 0u;
  double kfreq = 0.0;                          // the pair's RoPE frequency (kernel arguments)
  if (!GQA && a.v_new != nullptr) {
    if (tid < DV / 8)
      pend_piece = *(reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v_new) + ((int64_t)b * a.G + g) * DV) + tid);
    if (tid < a.d_r / 2) {
      pend_kbits = *reinterpret_cast<const uint32_t*>(static_cast<const uint16_t*>(a.kr_new) + (int64_t)b * a.d_r + 2 * tid);
      kfreq = p.inv_freq[tid];
    }
  }
  // The query: raw bf16 (GQA baseline); pre-absorbed fp32 (q_abs, q_rot);
  // or, fused, the raw positional pair and the first round of q / M_h
  // chunks for this wave's first head.
  u32x4 xqg[GQA ? NC : 1];
  f32x4 xa[GQA ? 1 : NC][2];
  f32x4 xr[NRC > 0 ? NRC : 1][2];
  const int W = a.d_c + a.d_r;
  // Fused absorption, q~[i] = sum_k q[k] M_h[i][k]: M_h is read in whole
  // rows, 16 lanes of 16 bytes per row and 4 rows per load, so each load
  // covers whole cache lines (the MFMA operand order, 64 bytes of 16 rows
  // per load, took four times as long to arrive).  Each lane forms an
  // 8-term bf16 dot product with its piece of q, and a DPP sum over the
  // row's 16 lanes finishes the row.  Columns come in segments of 128, rows
  // in blocks of 4 AR: one load round per (segment, row block).  Loads are
  // unconditional, from clamped addresses (selecting a loaded value would
  // wait for it and for every load before it); pieces past d_c meet a
  // zeroed query piece.
  constexpr int ARB = DV / 4 / AR;             // row blocks per segment
  u32x4 am[FUSED ? AR : 1];
  u32x4 xqf = {0u, 0u, 0u, 0u};                // the query piece of the lane's columns
  const int nrounds = ((a.d_c + 127) / 128) * ARB;
  const int a_row = lane >> 4, a_col = 8 * (lane & 15);
  const int npair = a.d_r / 2;
  const int ptid = NT - 1 - tid;
  const bool has_pair = FUSED && ptid < HPG * npair;
  const int pair_h = npair > 0 ? ptid / npair : 0, pair_i = npair > 0 ? ptid % npair : 0;
  uint32_t rq_bits = 0u;                       // the raw positional pair (bf16 x 2)
  double qfreq = 0.0;
  auto load_round = [&](int hl, int ro) {      // the query piece and M_h pieces of one round
    const int h = h0 + hl;
    const int col = min((ro / ARB) * 128 + a_col, a.d_c - 8), rb = ro % ARB;
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + ((int64_t)b * a.H + h) * W;
    const uint16_t* mh = static_cast<const uint16_t*>(a.m) + ((int64_t)h * DV + rb * AR * 4 + a_row) * a.d_c + col;
    xqf = *reinterpret_cast<const u32x4*>(qrow + col);
#pragma unroll
    for (int r = 0; r < AR; ++r) am[r] = *reinterpret_cast<const u32x4*>(mh + (int64_t)(4 * r) * a.d_c);
  };
  if constexpr (GQA) {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + ((int64_t)b * a.H + hq) * a.q_stride + 8 * qd;
#pragma unroll
    for (int c = 0; c < NC; ++c) xqg[c] = *reinterpret_cast<const u32x4*>(qrow + 32 * c);
  } else if constexpr (!FUSED) {
    const float* qa = a.q_abs + ((int64_t)b * a.H + hq) * DV + 8 * qd;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      xa[c][0] = *reinterpret_cast<const f32x4*>(qa + 32 * c);
      xa[c][1] = *reinterpret_cast<const f32x4*>(qa + 32 * c + 4);
    }
#pragma unroll
    for (int rc = 0; rc < NRC; ++rc) {
      const int j0 = min(32 * rc + 8 * qd, a.d_r - 8);    // lanes past d_r: any valid piece
      const float* qr = a.q_rot + ((int64_t)b * a.H + hq) * a.d_r + j0;
      xr[rc][0] = *reinterpret_cast<const f32x4*>(qr);
      xr[rc][1] = *reinterpret_cast<const f32x4*>(qr + 4);
    }
  } else {
    if (has_pair) {
      rq_bits = *reinterpret_cast<const uint32_t*>(
          static_cast<const uint16_t*>(a.q) + ((int64_t)b * a.H + h0 + pair_h) * W + a.d_c + 2 * pair_i);
      qfreq = p.inv_freq[pair_i];
    }
    if (w < HPG) load_round(w, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (!settle_rows()) {
    write_empty();
    return;
  }

  // Paged: the page ids of the split's rows [r0, r1), clamped into the pool
  // (an id outside it reads some page's data but never outside the pool).
  const int PR = PAGED ? a.page_rows : 1;
  const int pg0 = r0 / PR;
  if constexpr (PAGED) {
    const int npg = (r1 + PR - 1) / PR - pg0;
    const int32_t* bt = a.block_table + (int64_t)b * a.max_pages + pg0;
    for (int i = tid; i < npg; i += NT) {
      const int id = bt[i];
      split_pages[i] = id < 0 ? 0 : (id >= a.n_pages ? a.n_pages - 1 : id);
    }
    __syncthreads();
  }

  // With the current token's rows given, the split holding row L-1 takes
  // that row from them and streams only the rows before it from the cache.
  const bool pending = !GQA && a.v_new != nullptr && L > 0 && r0 <= L - 1 && L - 1 < r1;
  if (pending) r1 = L - 1;
  const int r1c = ((r1 + kLayoutRows - 1) / kLayoutRows) * kLayoutRows;

  // ---- streaming setup.  Rows are read through buffer descriptors that end
  // at the split's last layout tile: a tile past the end reads as zeros
  // without touching memory, so prefetches are issued unconditionally (the
  // wait counts stay static) and cost no traffic.  Each load is addressed as
  // a loop-invariant per-lane offset plus the tile base in a scalar
  // register.  Rows past the split inside its last layout tile may hold
  // never-written data; the tail tile zeroes them before use.
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + ((int64_t)b * a.G + g) * a.t_max * DV;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.kr) + (int64_t)b * a.t_max * a.d_r;
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(vbase), (short)0, r1c * DV * 2, kBufferWord3);
  const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(kbase), (short)0, r1c * a.d_r * 2, kBufferWord3);
  const __amdgpu_buffer_rsrc_t kcres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(GQA ? static_cast<const void*>(static_cast<const uint16_t*>(a.k_gqa) +
                                                       ((int64_t)b * a.G + g) * a.t_max * DV)
                            : static_cast<const void*>(vbase)),
      (short)0, r1c * DV * 2, kBufferWord3);
  const int kpieces = a.d_r / 8;              // 16-byte pieces per key row
  const int v_lane = qd * 256 + n * 16;       // piece qd of row n (of a 32-column chunk)
  int k_lane[NRC > 0 ? NRC : 1];
#pragma unroll
  for (int rc = 0; rc < NRC; ++rc)            // lanes past d_r re-read a valid piece (weight 0)
    k_lane[rc] = min(4 * rc + qd, kpieces - 1) * 256 + n * 16;
  const int v_tile_bytes = 16 * DV * 2, k_tile_bytes = 16 * a.d_r * 2;

  const int ntiles = (r1 - r0 + kTileRows - 1) / kTileRows;
  const int my_tiles = ntiles > w ? (ntiles - w + NW - 1) / NW : 0;
  auto tile_row = [&](int j) { return r0 + (w + NW * j) * kTileRows; };
  // Paged: the descriptors of the page holding a tile (a tile never spans
  // pages: pages are whole multiples of 32 rows), ending at the split's last
  // layout tile like the contiguous ones; a tile past it gets empty ones.
  auto page_res = [&](int row0, __amdgpu_buffer_rsrc_t& vr, __amdgpu_buffer_rsrc_t& kr, int& lt) {
    const int pg = row0 / PR;
    const bool live = row0 < r1c;
    const int page = live ? __builtin_amdgcn_readfirstlane(split_pages[pg - pg0]) : 0;
    const int rows = live ? min(PR, r1c - pg * PR) : 0;
    const uint16_t* vp = static_cast<const uint16_t*>(a.v) + ((int64_t)page * a.G + g) * PR * DV;
    const uint16_t* kp = static_cast<const uint16_t*>(a.kr) + (int64_t)page * PR * a.d_r;
    vr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vp), (short)0, rows * DV * 2, kBufferWord3);
    kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kp), (short)0, rows * a.d_r * 2, kBufferWord3);
    lt = (row0 - pg * PR) / kLayoutRows;
  };
  auto load_tile = [&](TileT& t, int row0) {
    int lt = row0 / kLayoutRows;               // first layout tile (uniform)
    __amdgpu_buffer_rsrc_t tv = vres, tk = kres;
    if constexpr (PAGED) page_res(row0, tv, tk, lt);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int vsoff = (lt + hf) * v_tile_bytes;
      if constexpr (GQA) {                     // keys first: the scores need them first
#pragma unroll
        for (int c = 0; c < NC; ++c)
          t.kc[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(kcres, v_lane + 1024 * c, vsoff, kAuxNT));
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
        t.v[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(tv, v_lane + 1024 * c, vsoff, kAuxNT));
      const int ksoff = (lt + hf) * k_tile_bytes;
#pragma unroll
      for (int rc = 0; rc < NRC; ++rc)
        t.k[hf][rc] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(tk, k_lane[rc], ksoff, KR_STREAM ? kAuxNT : 0));
    }
  };
  TileT buf[DEPTH];
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d) {
    load_tile(buf[d], tile_row(d));
    __builtin_amdgcn_sched_barrier(0);
  }

  // ---- the current token's rows (Algorithm 1's append): wave 0 rotates
  // the positional pair (fp64 angle, one rounding, exactly as append_kernel
  // does), stages the row in LDS for the epilogue and stores it into the
  // caches.  This workgroup is the only reader of row L-1 of stream (b, g)
  // in this launch; the shared positional key is stored once, by group 0.
  // Other workgroups may load the layout tile holding it, but only as rows
  // past their split, which are zeroed.  Run while the query loads land
  // (pre-absorbed path) or after the absorption (fused path, whose M_h
  // round holds too many registers to overlap it).
  auto stage_current_row = [&]() {
    if (!(pending && w == 0)) return;
    // row L-1 of stream (b, g), or, paged, row (L-1) mod page_rows of its page
    int64_t vs = ((int64_t)b * a.G + g) * a.t_max * DV, ks = (int64_t)b * a.t_max * a.d_r;
    int crow = L - 1;
    if constexpr (PAGED) {
      const int page = split_pages[(L - 1) / PR - pg0];
      vs = ((int64_t)page * a.G + g) * PR * DV;
      ks = (int64_t)page * PR * a.d_r;
      crow = (L - 1) % PR;
    }
    uint16_t* vcache = static_cast<uint16_t*>(a.v) + vs;
    uint16_t* kcache = static_cast<uint16_t*>(a.kr) + ks;
    if (tid < DV / 8) {
      *(reinterpret_cast<u32x4*>(prow) + tid) = pend_piece;
      *reinterpret_cast<u32x4*>(vcache + tiled_off<uint16_t>(crow, 8 * tid, DV)) = pend_piece;
    }
    if (tid < 16 * NRC) {
      uint16_t y0b = 0, y1b = 0;
      if (tid < a.d_r / 2) {
        double y0, y1;
        rotate_pair(bf16_bits_to_f32(pend_kbits & 0xFFFFu), bf16_bits_to_f32(pend_kbits >> 16),
                    (double)(L - 1) * kfreq, y0, y1);
        y0b = f64_to_bf16_rne(y0);
        y1b = f64_to_bf16_rne(y1);
        if (g == 0) {
          const int64_t o = tiled_off<uint16_t>(crow, 2 * tid, a.d_r);
          kcache[o] = y0b;
          kcache[o + 1] = y1b;
        }
      }
      prow[DV + 2 * tid] = y0b;
      prow[DV + 2 * tid + 1] = y1b;
    }
  };

  // ---- the query as MFMA B operands: absorbed, rotated and scaled, each
  // head's values split into bf16 high and low columns.
  bf16x8 bq[NC];
  bf16x8 bk[NRC > 0 ? NRC : 1];
  if constexpr (GQA) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float x[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[2 * j] = bf16_bits_to_f32(xqg[c][j] & 0xFFFFu) * a.scale_log2;
        x[2 * j + 1] = bf16_bits_to_f32(xqg[c][j] >> 16) * a.scale_log2;
      }
      bq[c] = active ? split_hi_lo(x, is_lo) : zero8;
    }
  } else if constexpr (!FUSED) {
    stage_current_row();
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float x[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = xa[c][0][j] * a.scale_log2;
        x[4 + j] = xa[c][1][j] * a.scale_log2;
      }
      bq[c] = active ? split_hi_lo(x, is_lo) : zero8;
    }
#pragma unroll
    for (int rc = 0; rc < NRC; ++rc) {
      const bool in_range = 32 * rc + 8 * qd < a.d_r;
      float x[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = xr[rc][0][j] * a.scale_log2;
        x[4 + j] = xr[rc][1][j] * a.scale_log2;
      }
      bk[rc] = (active && in_range) ? split_hi_lo(x, is_lo) : zero8;
    }
  } else {
    // Fused absorption, wave w taking heads w, w+4, ...: each round's rows
    // are finished by a sum over their lanes and stored (first segment) or
    // added (later segments) by the row's first lane, pre-scaled.  The first
    // round was loaded above.
    float* qs = lds;                                  // [HPG][QS_STRIDE]
    float* qrs = lds + HPG * Cfg::QS_STRIDE;          // [HPG][QR_STRIDE]
    auto absorb_round = [&](int hl, int ro) {
      const int rb = ro % ARB;
      const u32x4 qv = (ro / ARB) * 128 + a_col < a.d_c ? xqf : u32x4{0u, 0u, 0u, 0u};
      float v[AR];
#pragma unroll
      for (int r = 0; r < AR; ++r) v[r] = dot8_bf16(am[r], qv);
#pragma unroll
      for (int r = 0; r < AR; ++r) v[r] = sum16(v[r]) * a.scale_log2;
      // every lane of a row's 16 writes the same value
      float* dst = qs + hl * Cfg::QS_STRIDE + rb * AR * 4 + a_row;
      if (ro < ARB) {
#pragma unroll
        for (int r = 0; r < AR; ++r) dst[4 * r] = v[r];
      } else {
#pragma unroll
        for (int r = 0; r < AR; ++r) dst[4 * r] += v[r];
      }
    };
    // the first round (loaded before the tiles) in straight-line code, so
    // its waits count only its own loads; then the rest
    if (w < HPG) absorb_round(w, 0);
    for (int hl = w; hl < HPG; hl += NW)
      for (int ro = hl == w ? 1 : 0; ro < nrounds; ++ro) {
        load_round(hl, ro);
        absorb_round(hl, ro);
      }
    stage_current_row();
    // rotate the positional query at position L-1 (fp64 angle, reduced
    // exactly, fp32 rotation); the padding past d_r is written as zeros in
    // the same phase, so one barrier covers both
    if (has_pair) {
      float y0, y1;
      rotate_query_pair(bf16_bits_to_f32(rq_bits & 0xFFFFu), bf16_bits_to_f32(rq_bits >> 16),
                        (double)(L > 0 ? L - 1 : 0) * qfreq, a.scale_log2, y0, y1);
      qrs[pair_h * Cfg::QR_STRIDE + 2 * pair_i] = y0;
      qrs[pair_h * Cfg::QR_STRIDE + 2 * pair_i + 1] = y1;
    }
    if constexpr (NRC > 0) {
      for (int idx = tid; idx < HPG * 32 * NRC; idx += NT) {
        const int j = idx % (32 * NRC);
        if (j >= a.d_r) qrs[(idx / (32 * NRC)) * Cfg::QR_STRIDE + j] = 0.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float* src = qs + col_head * Cfg::QS_STRIDE + 32 * c + 8 * qd;
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = src[j];
      bq[c] = active ? split_hi_lo(x, is_lo) : zero8;
    }
#pragma unroll
    for (int rc = 0; rc < NRC; ++rc) {
      const float* src = qrs + col_head * Cfg::QR_STRIDE + 32 * rc + 8 * qd;
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = src[j];
      bk[rc] = active ? split_hi_lo(x, is_lo) : zero8;
    }
  }

  // identity selectors for the V transpose: E_half[k][n] = (k == n + 16 half)
  bf16x8 esel[2];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    u32x4 u = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (8 * qd + j == n + 16 * half) u[j >> 1] |= 0x3F80u << (16 * (j & 1));
    esel[half] = as_bf16x8(u);
  }

  // ---- streaming loop
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int ib = 0; ib < NB; ++ib) acc[ib] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute_tile = [&](TileT& t, int row0, int row_end) {
    if (row0 + kTileRows > row_end) {        // ragged tail: clear rows past the end
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bool dead = row0 + 16 * hf + n >= row_end;
#pragma unroll
        for (int c = 0; c < NC; ++c) t.v[hf][c] = dead ? zero8 : t.v[hf][c];
        if constexpr (GQA) {
#pragma unroll
          for (int c = 0; c < NC; ++c) t.kc[hf][c] = dead ? zero8 : t.kc[hf][c];
        }
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc) t.k[hf][rc] = dead ? zero8 : t.k[hf][rc];
      }
    }
    // scores: rows 16*hf + 4*qd + jj of the tile, column n
    f32x4 sc[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      sc[hf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) sc[hf] = mfma16(GQA ? t.kc[hf][c] : t.v[hf][c], bq[c], sc[hf]);
#pragma unroll
      for (int rc = 0; rc < NRC; ++rc) sc[hf] = mfma16(t.k[hf][rc], bk[rc], sc[hf]);
    }
    float x[8];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const float v = sc[hf][jj];
        x[4 * hf + jj] = v + mirror<HPG>(v);   // hi + lo part of the same head
      }
    if (row0 + kTileRows > row_end) {        // ragged tail: rows past the end
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (row0 + 16 * (k >> 2) + 4 * qd + (k & 3) >= row_end) x[k] = -INFINITY;
    }
    float mt = x[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) mt = fmaxf(mt, x[k]);
    mt = max_over_rows(mt);
    const float m_new = fmaxf(m_run, mt);
    if (__ballot(m_new > m_run) != 0) {      // rescale only when a max grew
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) acc[ib] *= alpha;
      m_run = m_new;
    }
    float pr[8];
    float psum = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      pr[k] = __builtin_amdgcn_exp2f(x[k] - m_run);
      psum += pr[k];
    }
    l_run += psum;
    const bf16x8 bp = active ? split_hi_lo(pr, is_lo) : zero8;
    // P.V: transpose each 16x16 block of V with an identity MFMA, then
    // accumulate O^T[i][n] over the tile's 32 rows.
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        const f32x4 t0 = mfma16(t.v[0][c], esel[half], z);
        const f32x4 t1 = mfma16(t.v[1][c], esel[half], z);
        bf16x8 a;
        const bf16x2 a01 = __builtin_convertvector((f32x2{t0[0], t0[1]}), bf16x2);
        const bf16x2 a23 = __builtin_convertvector((f32x2{t0[2], t0[3]}), bf16x2);
        const bf16x2 a45 = __builtin_convertvector((f32x2{t1[0], t1[1]}), bf16x2);
        const bf16x2 a67 = __builtin_convertvector((f32x2{t1[2], t1[3]}), bf16x2);
        a[0] = a01[0]; a[1] = a01[1]; a[2] = a23[0]; a[3] = a23[1];
        a[4] = a45[0]; a[5] = a45[1]; a[6] = a67[0]; a[7] = a67[1];
        acc[2 * c + half] = mfma16(a, bp, acc[2 * c + half]);
      }
  };

  // DEPTH-stage register pipeline: tile j+DEPTH-1 is requested before tile
  // j is consumed.  Every iteration issues the same loads, so the waits the
  // compiler places are exact; the scheduling barrier keeps each tile's
  // loads in issue order, so the oldest tile is always the first to land.
  for (int jt = 0; jt < my_tiles; jt += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int j = jt + d;
      if (j >= my_tiles) break;
      load_tile(buf[(d + DEPTH - 1) % DEPTH], tile_row(j + DEPTH - 1));
      __builtin_amdgcn_sched_barrier(0);
      compute_tile(buf[d], tile_row(j), r1);
    }
  }

  // ---- the current token's row, staged in LDS by wave 0 in the prologue,
  // scored by wave 0 as a one-row tile
  if (pending && w == 0) {
    TileT t;
    const u32x4* pv = reinterpret_cast<const u32x4*>(prow);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      t.v[0][c] = n == 0 ? as_bf16x8(pv[4 * c + qd]) : zero8;
      t.v[1][c] = zero8;
    }
#pragma unroll
    for (int rc = 0; rc < NRC; ++rc) {
      t.k[0][rc] = n == 0 ? as_bf16x8(pv[DV / 8 + 4 * rc + qd]) : zero8;
      t.k[1][rc] = zero8;
    }
    compute_tile(t, L - 1, L);
  }

  // ---- merge the waves and write this split's partial
  l_run = sum_over_rows(l_run);
#pragma unroll
  for (int ib = 0; ib < NB; ++ib)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) acc[ib][jj] += mirror<HPG>(acc[ib][jj]);

  __syncthreads();   // the prologue's LDS is reused below
  constexpr int RS = DV + 2;                     // per-(wave, head) record: [m, l, o[DV]]
  float* red = lds;
  if (n < HPG) {
    float* rec = red + (w * HPG + n) * RS;
    if (qd == 0) {
      rec[0] = m_run;
      rec[1] = l_run;
    }
#pragma unroll
    for (int ib = 0; ib < NB; ++ib)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) rec[2 + 16 * ib + 4 * qd + jj] = acc[ib][jj];
  }
  __syncthreads();
  for (int idx = tid; idx < HPG * DV; idx += NT) {
    const int hl = idx / DV, i = idx % DV;
    float mx = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) mx = fmaxf(mx, red[(ww * HPG + hl) * RS]);
    float o = 0.f, lsum = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) {
        const float* rec = red + (ww * HPG + hl) * RS;
        const float sc = rec[0] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(rec[0] - mx);
        lsum += rec[1] * sc;
        o += rec[2 + i] * sc;
      }
      o /= lsum;
    }
    const int64_t prow = ((int64_t)b * a.H + h0 + hl) * a.S + s;
    a.o_part[prow * DV + i] = o;
    if (i == 0) a.lse_part[prow] = mx == -INFINITY ? -INFINITY : (mx + log2f(lsum)) * kLn2;
  }
}

// ========================================================== decode (f32)
// Vector-ALU variant for fp32 storage.  Per 64-row tile a wave first scores
// one row per lane, then accumulates the weighted rows with one output
// element per lane.
constexpr int kF32MaxHpg = 8;
constexpr int kF32MaxDv = 256;
constexpr int kF32MaxDr = 64;

__global__ void __launch_bounds__(kThreads) decode_f32_kernel(DecodeParams p) {
  __shared__ float qs[kF32MaxHpg][kF32MaxDv + 1];
  __shared__ float qr[kF32MaxHpg][kF32MaxDr];
  __shared__ float pb[kWaves][64][kF32MaxHpg];
  __shared__ float red_ml[kWaves][kF32MaxHpg][2];
  __shared__ float red_o[kWaves][kF32MaxHpg][kF32MaxDv];

  int b, s, g;
  bool empty_slot;
  if (!work_item(p.a, b, s, g, empty_slot)) return;   // grid padding
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int hpg = p.a.H / p.a.G, h0 = g * hpg;
  const int DV = p.a.d_v, DR = p.a.d_r;
  const int L = clamp_len(p.a.lens, b, p.a.t_max);
  int r0, r1;
  split_rows(L, p.a.S, p.a.split_rows, s, r0, r1);
  if (r0 >= r1 && s > 0) {                     // an empty split past the first: lse only
    if (tid < hpg) p.a.lse_part[((int64_t)b * p.a.H + h0 + tid) * p.a.S + s] = -INFINITY;
    return;
  }
  const bool pending = p.a.v_new != nullptr && L > 0 && r0 <= L - 1 && L - 1 < r1;
  if (pending) r1 = L - 1;

  if (p.a.fused) {
    const float* qg = static_cast<const float*>(p.a.q);
    const float* mg = static_cast<const float*>(p.a.m);
    const int W = p.a.d_c + DR;
    for (int idx = tid; idx < hpg * DV; idx += kThreads) {
      const int hl = idx / DV, i = idx % DV;
      const float* qrow = qg + ((int64_t)b * p.a.H + h0 + hl) * W;
      const float* mrow = mg + ((int64_t)(h0 + hl) * DV + i) * p.a.d_c;
      const float a = dot_f32(qrow, mrow, p.a.d_c);
      qs[hl][i] = a * p.a.scale_log2;
    }
    const int L1 = L > 0 ? L - 1 : 0;
    for (int idx = tid; idx < hpg * (DR / 2); idx += kThreads) {
      const int hl = idx / (DR / 2), i = idx % (DR / 2);
      const float* qrow = qg + ((int64_t)b * p.a.H + h0 + hl) * W + p.a.d_c;
      double y0, y1;
      rotate_pair(qrow[2 * i], qrow[2 * i + 1], (double)L1 * p.inv_freq[i], y0, y1);
      qr[hl][2 * i] = (float)(y0 * (double)p.a.scale_log2);
      qr[hl][2 * i + 1] = (float)(y1 * (double)p.a.scale_log2);
    }
  } else {
    for (int idx = tid; idx < hpg * DV; idx += kThreads) {
      const int hl = idx / DV, i = idx % DV;
      qs[hl][i] = p.a.q_abs[((int64_t)b * p.a.H + h0 + hl) * DV + i] * p.a.scale_log2;
    }
    for (int idx = tid; idx < hpg * DR; idx += kThreads) {
      const int hl = idx / DR, j = idx % DR;
      qr[hl][j] = p.a.q_rot[((int64_t)b * p.a.H + h0 + hl) * DR + j] * p.a.scale_log2;
    }
  }
  __syncthreads();

  const float* vb = static_cast<const float*>(p.a.v) + ((int64_t)b * p.a.G + g) * p.a.t_max * DV;
  const float* kb = static_cast<const float*>(p.a.kr) + (int64_t)b * p.a.t_max * DR;
  float m_run[kF32MaxHpg], l_run[kF32MaxHpg], acc[kF32MaxHpg][4];
#pragma unroll
  for (int h = 0; h < kF32MaxHpg; ++h) {
    m_run[h] = -INFINITY;
    l_run[h] = 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[h][u] = 0.f;
  }
  const int ntiles = (r1 - r0 + 63) / 64;
  const int iters = (ntiles + kWaves - 1) / kWaves;
  for (int it = 0; it < iters; ++it) {
    const int tile = w + kWaves * it;
    const int row0 = r0 + 64 * tile;
    const bool has = tile < ntiles;
    if (has) {
      const int t = row0 + lane;
      const bool valid = t < r1;
      float sc[kF32MaxHpg];
#pragma unroll
      for (int h = 0; h < kF32MaxHpg; ++h) sc[h] = 0.f;
      if (valid) {
        // the row's 16-byte pieces (4 floats each, contiguous in the tiled
        // layout), eight requested per step
        const float* vrow = vb + tiled_off<float>(t, 0, DV);
        const int npc = DV / 4;
        for (int pc0 = 0; pc0 < npc; pc0 += 8) {
          f32x4 vv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u)
            vv[u] = pc0 + u < npc ? *reinterpret_cast<const f32x4*>(vrow + (int64_t)(pc0 + u) * 4 * kLayoutRows)
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            if (pc0 + u >= npc) break;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int i = 4 * (pc0 + u) + e;
#pragma unroll
              for (int h = 0; h < kF32MaxHpg; ++h)
                if (h < hpg) sc[h] = fmaf(qs[h][i], vv[u][e], sc[h]);
            }
          }
        }
        const float* krow = kb + tiled_off<float>(t, 0, DR);
        for (int pc0 = 0; pc0 < DR / 4; pc0 += 8) {
          f32x4 kv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u)
            kv[u] = pc0 + u < DR / 4 ? *reinterpret_cast<const f32x4*>(krow + (int64_t)(pc0 + u) * 4 * kLayoutRows)
                                     : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            if (pc0 + u >= DR / 4) break;
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
              for (int h = 0; h < kF32MaxHpg; ++h)
                if (h < hpg) sc[h] = fmaf(qr[h][4 * (pc0 + u) + e], kv[u][e], sc[h]);
          }
        }
      }
#pragma unroll
      for (int h = 0; h < kF32MaxHpg; ++h) {
        if (h < hpg) {
          const float x = valid ? sc[h] : -INFINITY;
          const float mt = wave_max(x);
          const float m_new = fmaxf(m_run[h], mt);
          const float alpha = __builtin_amdgcn_exp2f(m_run[h] - m_new);
          const float pr = __builtin_amdgcn_exp2f(x - m_new);
          l_run[h] = l_run[h] * alpha + wave_sum(pr);
#pragma unroll
          for (int u = 0; u < 4; ++u) acc[h][u] *= alpha;
          m_run[h] = m_new;
          pb[w][lane][h] = pr;
        }
      }
    }
    __syncthreads();
    if (has) {
      const int nrow = r1 - row0 < 64 ? r1 - row0 : 64;
#pragma unroll 16
      for (int t = 0; t < nrow; ++t) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = lane + 64 * u;
          if (i < DV) {
            const float v = vb[tiled_off<float>(row0 + t, i, DV)];
#pragma unroll
            for (int h = 0; h < kF32MaxHpg; ++h)
              if (h < hpg) acc[h][u] = fmaf(pb[w][t][h], v, acc[h][u]);
          }
        }
      }
    }
    __syncthreads();
  }

  // the pending row (current token), taken from v_new / kr_new with the
  // rotation and rounding gva_append_kv would store, added by wave 0
  if (pending && w == 0) {
    const float* vn = static_cast<const float*>(p.a.v_new) + ((int64_t)b * p.a.G + g) * DV;
    float vv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) vv[u] = lane + 64 * u < DV ? vn[lane + 64 * u] : 0.f;
    float kk = 0.f;
    if (lane < DR) {
      const float* kn = static_cast<const float*>(p.a.kr_new) + (int64_t)b * DR;
      double y0, y1;
      const int pi = lane / 2;
      rotate_pair(kn[2 * pi], kn[2 * pi + 1], (double)(L - 1) * p.inv_freq[pi], y0, y1);
      kk = (float)((lane & 1) ? y1 : y0);
    }
    // the append of row L-1 (this wave is its only reader in this launch)
    float* vcache = static_cast<float*>(p.a.v) + ((int64_t)b * p.a.G + g) * p.a.t_max * DV;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (lane + 64 * u < DV) vcache[tiled_off<float>(L - 1, lane + 64 * u, DV)] = vv[u];
    if (g == 0 && lane < DR)
      (static_cast<float*>(p.a.kr) + (int64_t)b * p.a.t_max * DR)[tiled_off<float>(L - 1, lane, DR)] = kk;
#pragma unroll
    for (int h = 0; h < kF32MaxHpg; ++h) {
      if (h < hpg) {
        float part = lane < DR ? qr[h][lane] * kk : 0.f;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (lane + 64 * u < DV) part = fmaf(qs[h][lane + 64 * u], vv[u], part);
        const float x = wave_sum(part);
        const float m_new = fmaxf(m_run[h], x);
        const float alpha = __builtin_amdgcn_exp2f(m_run[h] - m_new);
        const float pr = __builtin_amdgcn_exp2f(x - m_new);
        l_run[h] = l_run[h] * alpha + pr;
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[h][u] = acc[h][u] * alpha + pr * vv[u];
        m_run[h] = m_new;
      }
    }
  }

#pragma unroll
  for (int h = 0; h < kF32MaxHpg; ++h) {
    if (h < hpg) {
      if (lane == 0) {
        red_ml[w][h][0] = m_run[h];
        red_ml[w][h][1] = l_run[h];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = lane + 64 * u;
        if (i < DV) red_o[w][h][i] = acc[h][u];
      }
    }
  }
  __syncthreads();
  for (int idx = tid; idx < hpg * DV; idx += kThreads) {
    const int hl = idx / DV, i = idx % DV;
    float mx = -INFINITY;
    for (int ww = 0; ww < kWaves; ++ww) mx = fmaxf(mx, red_ml[ww][hl][0]);
    float o = 0.f, lsum = 0.f;
    if (mx != -INFINITY) {
      for (int ww = 0; ww < kWaves; ++ww) {
        const float mw = red_ml[ww][hl][0];
        const float sc = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - mx);
        lsum += red_ml[ww][hl][1] * sc;
        o += red_o[ww][hl][i] * sc;
      }
      o /= lsum;
    }
    const int64_t prow = ((int64_t)b * p.a.H + h0 + hl) * p.a.S + s;
    p.a.o_part[prow * DV + i] = o;
    if (i == 0) p.a.lse_part[prow] = mx == -INFINITY ? -INFINITY : (mx + log2f(lsum)) * kLn2;
  }
}

// =============================================================== combine
// One wave per (b, h) row, lane = output element (up to 4 per lane).  A
// single pass keeps a running log-sum-exp and rescales the running sum;
// the split loads do not depend on each other, so they overlap.
constexpr int kCombineMaxDv = 256;
constexpr long long kChunkItemsPerCu = 2;         // bounded chunks: chunks per CU
constexpr long long kMinChunkBytes = 128 << 10;   // bounded chunks: value bytes per chunk
constexpr long long kMinSplitStream = 192 << 10;  // even splits: a stream's value bytes worth splitting
constexpr long long kMinSplitBytes = 32 << 10;    // even splits: value bytes per split
constexpr long long kMaxEvenSplits = 16;

__global__ void __launch_bounds__(kThreads) combine_kernel(CombineParams p) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (row >= p.rows) return;
  const float* lp = p.lse_part + (int64_t)row * p.S;
  const float* op = p.o_part + (int64_t)row * p.S * p.d_v;
  // the row's split LSEs, up to 4 per lane (S <= 256), and their maximum
  float l[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int s = lane + 64 * k;
    l[k] = s < p.S ? lp[s] : -INFINITY;
  }
  // The first kSpec splits' partials are requested with the LSEs, before it
  // is known which are empty (splits hold a sequence's rows from the front,
  // so the first ones are the likely non-empty ones): one memory round trip
  // less.  Empty splits' values are loaded but never used (selected away,
  // so whatever they hold cannot reach the output).
  constexpr int kSpec = 8;
  float v0[kSpec][4];
#pragma unroll
  for (int j = 0; j < kSpec; ++j)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = lane + 64 * u;
      v0[j][u] = (j < p.S && i < p.d_v) ? op[(int64_t)j * p.d_v + i] : 0.f;
    }
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < 4; ++k) mx = fmaxf(mx, l[k]);
  mx = wave_max(mx);
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  float z = 0.f;
  if (mx != -INFINITY) {
    float wk[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      wk[k] = l[k] == -INFINITY ? 0.f : expf(l[k] - mx);
      z += wk[k];
    }
    z = wave_sum(z);
#pragma unroll
    for (int j = 0; j < kSpec; ++j) {
      if (j >= p.S) break;
      const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wk[0]), j));
      const bool live = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(l[0]), j)) != -INFINITY;
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] = live ? fmaf(wj, v0[j][u], acc[u]) : acc[u];
    }
    // the remaining splits with rows, 8 at a time so their loads overlap
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (64 * k >= p.S) break;
      unsigned long long mask = __ballot(l[k] != -INFINITY);
      if (k == 0) mask &= ~((1ull << kSpec) - 1ull);
      while (mask != 0ull) {
        int sel[8];
        float wsel[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          sel[j] = -1;
          wsel[j] = 0.f;
          if (mask != 0ull) {
            const int bit = __builtin_ctzll(mask);
            mask &= mask - 1ull;
            sel[j] = 64 * k + bit;
            wsel[j] = __shfl(wk[k], bit, 64);
          }
        }
        float v[8][4];
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int i = lane + 64 * u;
            v[j][u] = (sel[j] >= 0 && i < p.d_v) ? op[(int64_t)sel[j] * p.d_v + i] : 0.f;
          }
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int u = 0; u < 4; ++u) acc[u] = fmaf(wsel[j], v[j][u], acc[u]);
      }
    }
  }
  const float inv = z > 0.f ? 1.f / z : 0.f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = lane + 64 * u;
    if (i < p.d_v) p.o[(int64_t)row * p.d_v + i] = acc[u] * inv;
  }
  if (p.lse != nullptr && lane == 0) p.lse[row] = mx == -INFINITY ? -INFINITY : mx + logf(z);
}

using DecodeFn = void (*)(DecodeParams);

template <int HPG, int DV, bool FUSED, bool PAGED>
DecodeFn pick_nrc(int nrc, bool kr_stream) {
  switch (nrc) {
    case 0: return decode_bf16_kernel<HPG, DV, 0, false, FUSED, PAGED>;
    case 1: return kr_stream ? decode_bf16_kernel<HPG, DV, 1, false, FUSED, PAGED, true>
                             : decode_bf16_kernel<HPG, DV, 1, false, FUSED, PAGED>;
    case 2: return kr_stream ? decode_bf16_kernel<HPG, DV, 2, false, FUSED, PAGED, true>
                             : decode_bf16_kernel<HPG, DV, 2, false, FUSED, PAGED>;
  }
  return nullptr;
}

template <int HPG, int DV>
DecodeFn pick_mode(int nrc, bool fused, bool paged, bool kr_stream) {
  if (paged) return fused ? pick_nrc<HPG, DV, true, true>(nrc, kr_stream) : pick_nrc<HPG, DV, false, true>(nrc, kr_stream);
  return fused ? pick_nrc<HPG, DV, true, false>(nrc, kr_stream) : pick_nrc<HPG, DV, false, false>(nrc, kr_stream);
}

template <int HPG>
DecodeFn pick_dv(int dv, int nrc, bool fused, bool paged, bool kr_stream) {
  switch (dv) {
    case 64: return pick_mode<HPG, 64>(nrc, fused, paged, kr_stream);
    case 128: return pick_mode<HPG, 128>(nrc, fused, paged, kr_stream);
  }
  return nullptr;
}

template <int DV>
DecodeFn pick_gqa_hpg(int hpg) {
  switch (hpg) {
    case 1: return decode_bf16_kernel<1, DV, 0, true, false, false>;
    case 2: return decode_bf16_kernel<2, DV, 0, true, false, false>;
    case 4: return decode_bf16_kernel<4, DV, 0, true, false, false>;
    case 8: return decode_bf16_kernel<8, DV, 0, true, false, false>;
  }
  return nullptr;
}

// Waves per GVA decode workgroup.  A launch with few workgroups leaves most
// CUs idle and is bound by each stream's chain of memory round trips, not
// by HBM: its workgroups take eight waves, so twice as many of each stream's
// tiles are in flight at once (one such workgroup per CU; sixteen waves
// would leave 128 registers per wave, too few for the tiles in flight).
// (The matched-GQA baseline, whose tiles carry a key row beside each value
// row, measured slower with eight waves at the 350M shape -- 14.5 against
// 13.2 us -- and keeps four.)
int decode_waves(long long grid, int n_cu) {
  return 2 * grid <= n_cu ? 8 : kWaves;
}

DecodeFn pick_gqa_decode(int hpg, int dv) {
  switch (dv) {
    case 64: return pick_gqa_hpg<64>(hpg);
    case 128: return pick_gqa_hpg<128>(hpg);
  }
  return nullptr;
}

// fused absorption, contiguous caches, NW waves (the few-workgroup launches)
template <int HPG, int DV, int NW>
DecodeFn pick_wide_nrc(int nrc) {
  switch (nrc) {
    case 0: return decode_bf16_kernel<HPG, DV, 0, false, true, false, false, NW>;
    case 1: return decode_bf16_kernel<HPG, DV, 1, false, true, false, false, NW>;
    case 2: return decode_bf16_kernel<HPG, DV, 2, false, true, false, false, NW>;
  }
  return nullptr;
}

template <int HPG>
DecodeFn pick_wide(int dv, int nrc, int nw) {
  switch (dv * 100 + nw) {
    case 6408: return pick_wide_nrc<HPG, 64, 8>(nrc);
    case 12808: return pick_wide_nrc<HPG, 128, 8>(nrc);
  }
  return nullptr;
}

DecodeFn pick_bf16_decode(int hpg, int dv, int nrc, bool fused, bool paged, bool kr_stream, int nw) {
  if (nw != kWaves) {
    if (!fused || paged) return nullptr;
    switch (hpg) {
      case 1: return pick_wide<1>(dv, nrc, nw);
      case 2: return pick_wide<2>(dv, nrc, nw);
      case 4: return pick_wide<4>(dv, nrc, nw);
      case 8: return pick_wide<8>(dv, nrc, nw);
    }
    return nullptr;
  }
  switch (hpg) {
    case 1: return pick_dv<1>(dv, nrc, fused, paged, kr_stream);
    case 2: return pick_dv<2>(dv, nrc, fused, paged, kr_stream);
    case 4: return pick_dv<4>(dv, nrc, fused, paged, kr_stream);
    case 8: return pick_dv<8>(dv, nrc, fused, paged, kr_stream);
  }
  return nullptr;
}

// The positional-key tiles are read by the G groups of a split through one
// L2, so they are normally cached.  With at least as many (sequence, group)
// streams as CUs, every L2 holds many sequences' keys at once and streaming
// them (non-temporal, like the value tiles) measured faster: B = 32, G = 8
// on 256 CUs gained 0.7-2.0 us per launch, while four long sequences
// (32 streams) lost 2.6-3 us.  Paged caches the same: 2.1-2.7 us per
// launch at B = 32, G = 8 with pages of 64 or 256 rows.
bool decode_kr_stream(const gva_dims* d) {
  return (long long)d->batch * d->n_groups >= device_cu_count();
}

// With launch = false every argument is checked and nothing is enqueued.
int absorb_impl(const gva_dims* dims, int n_per_seq, const void* q, const void* m, const int32_t* lens,
                float* q_abs, float* q_rot, void* stream, bool launch = true) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (n_per_seq < 1) return GVA_ERR_INVALID_ARG;
  if (!q || !m || !lens || !q_abs) return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && !q_rot) return GVA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(m, 16) || !aligned(lens, 4) || !aligned(q_abs, 16) ||
      (q_rot && !aligned(q_rot, 4)))
    return GVA_ERR_INVALID_ARG;
  if (dims->d_r / 2 > kMaxPairs) return GVA_ERR_UNSUPPORTED;
  const long long rows = (long long)dims->batch * n_per_seq;
  if (rows > (1LL << 20) || rows * dims->n_heads > 0x7FFFFFFFLL) return GVA_ERR_UNSUPPORTED;
  AbsorbParams p{};
  p.q = q;
  p.m = m;
  p.lens = lens;
  p.q_abs = q_abs;
  p.q_rot = q_rot;
  p.B = (int32_t)rows;
  p.H = dims->n_heads;
  p.d_v = dims->d_v;
  p.d_c = dims->d_c;
  p.d_r = dims->d_r;
  p.t_max = dims->t_max;
  p.n_per_seq = n_per_seq;
  // many rows (a prompt): each workgroup reuses M_h over 64 rows (32 from
  // 1024 rows on), which cuts the re-reads of M_h fourfold (twofold); a
  // decode batch keeps 16 rows per workgroup.  (2048 prompt rows at H = 16,
  // d = 64: 16.0 -> 10.3-11.1 us against one row block.)
  p.row_blocks = rows >= 2048 ? 4 : (rows >= 1024 ? 2 : 1);
  fill_inv_freq(dims, p.inv_freq);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dims->dtype == GVA_DTYPE_BF16 && (dims->d_v % 16 != 0 || dims->d_c % 32 != 0 || dims->d_r % 8 != 0))
    return GVA_ERR_UNSUPPORTED;
  if (!launch) return GVA_OK;
  if (dims->dtype == GVA_DTYPE_BF16) {
    const long long rows_per_wg = 16LL * p.row_blocks;
    const dim3 grid(dims->n_heads, (unsigned)((rows + rows_per_wg - 1) / rows_per_wg));
    hipLaunchKernelGGL(absorb_bf16_kernel, grid, dim3(kThreads), 0, s, p);
  } else {
    hipLaunchKernelGGL(absorb_f32_kernel, dim3((unsigned)(rows * dims->n_heads)), dim3(128), 0, s, p);
  }
  return launch_status();
}

int append_impl(const gva_dims* dims, const gva_paging* paging, const int32_t* block_table, void* v_cache,
                void* kr_cache, const void* v_new, const void* kr_new, const int32_t* seq, const int32_t* pos,
                int32_t n_rows, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (n_rows < 0) return GVA_ERR_INVALID_ARG;
  if (n_rows == 0) return GVA_OK;
  if (!v_cache || !v_new || !seq || !pos) return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && (!kr_cache || !kr_new)) return GVA_ERR_INVALID_ARG;
  if (!aligned(v_cache, 16) || !aligned(v_new, 16) || !aligned(seq, 4) || !aligned(pos, 4))
    return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && (!aligned(kr_cache, 16) || !aligned(kr_new, 4))) return GVA_ERR_INVALID_ARG;
  st = check_cache_layout(dims);
  if (st != GVA_OK) return st;
  AppendParams p{};
  p.v_cache = v_cache;
  p.kr_cache = kr_cache;
  p.v_new = v_new;
  p.kr_new = kr_new;
  p.seq = seq;
  p.pos = pos;
  p.B = dims->batch;
  p.G = dims->n_groups;
  p.t_max = dims->t_max;
  p.d_v = dims->d_v;
  p.d_r = dims->d_r;
  p.n_rows = n_rows;
  p.block_table = block_table;
  p.page_rows = paging ? paging->page_rows : 0;
  p.max_pages = paging ? paging->max_pages : 0;
  p.n_pages = paging ? paging->n_pages : 0;
  fill_inv_freq(dims, p.inv_freq);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dims->dtype == GVA_DTYPE_BF16)
    hipLaunchKernelGGL(append_kernel<uint16_t>, dim3(n_rows), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(append_kernel<float>, dim3(n_rows), dim3(256), 0, s, p);
  return launch_status();
}

// A paging description consistent with dims: pages of whole 32-row tiles,
// a block-table row covering the capacity exactly, ids for at most
// kMaxPages pages per sequence.
int check_paging(const gva_dims* dims, const gva_paging* pg, const int32_t* block_table) {
  if (pg == nullptr || block_table == nullptr || !aligned(block_table, 4)) return GVA_ERR_INVALID_ARG;
  if (pg->page_rows < kTileRows || pg->page_rows % kTileRows != 0) return GVA_ERR_INVALID_ARG;
  if (pg->max_pages < 1 || pg->n_pages < 1) return GVA_ERR_INVALID_ARG;
  if ((long long)pg->max_pages * pg->page_rows != dims->t_max) return GVA_ERR_INVALID_ARG;
  if (pg->max_pages > kMaxPages) return GVA_ERR_UNSUPPORTED;
  if (dims->dtype != GVA_DTYPE_BF16) return GVA_ERR_UNSUPPORTED;
  return GVA_OK;
}

// The attention launch behind gva_decode_attention and, with paging given,
// gva_paged_decode_attention (v_cache / kr_cache are then the page pools).
int decode_attention_impl(const gva_dims* dims, const gva_paging* paging, const int32_t* block_table,
                          const void* q, const void* m, const float* q_abs, const float* q_rot,
                          void* v_cache, void* kr_cache, const int32_t* lens, const void* v_new,
                          const void* kr_new, int32_t num_splits, int32_t split_rows, float* o_part,
                          float* lse_part, void* stream, bool launch = true) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS) return GVA_ERR_INVALID_ARG;
  if (split_rows < 0 || split_rows % kTileRows != 0) return GVA_ERR_INVALID_ARG;
  const bool fused = q != nullptr || m != nullptr;
  if (fused) {
    if (!q || !m || q_abs || q_rot) return GVA_ERR_INVALID_ARG;
    if (!aligned(q, 16) || !aligned(m, 16)) return GVA_ERR_INVALID_ARG;
  } else {
    if (!q_abs || (dims->d_r > 0 && !q_rot)) return GVA_ERR_INVALID_ARG;
    if (!aligned(q_abs, 16) || (q_rot && !aligned(q_rot, 16))) return GVA_ERR_INVALID_ARG;
  }
  if (!v_cache || !lens || !o_part || !lse_part) return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && !kr_cache) return GVA_ERR_INVALID_ARG;
  if (!aligned(v_cache, 16) || !aligned(lens, 4) || !aligned(o_part, 16) || !aligned(lse_part, 4) ||
      (dims->d_r > 0 && !aligned(kr_cache, 16)))
    return GVA_ERR_INVALID_ARG;
  if (!v_new && kr_new) return GVA_ERR_INVALID_ARG;          // the pending row comes whole
  if (v_new && (!aligned(v_new, 16) || (dims->d_r > 0 && (!kr_new || !aligned(kr_new, 4)))))
    return GVA_ERR_INVALID_ARG;
  st = check_cache_layout(dims);
  if (st != GVA_OK) return st;

  const int hpg = dims->n_heads / dims->n_groups;
  const long long n_items = decode_grid(dims, num_splits, split_rows);
  if (n_items > 0x7FFFFFFFLL) return GVA_ERR_UNSUPPORTED;

  DecodeParams p{};
  p.a.q = q;
  p.a.m = m;
  p.a.q_abs = q_abs;
  p.a.q_rot = q_rot;
  p.a.v = v_cache;
  p.a.kr = kr_cache;
  p.a.lens = lens;
  p.a.o_part = o_part;
  p.a.lse_part = lse_part;
  p.a.v_new = v_new;
  p.a.kr_new = kr_new;
  p.a.k_gqa = nullptr;
  p.a.q_stride = 0;
  p.a.B = dims->batch;
  p.a.H = dims->n_heads;
  p.a.G = dims->n_groups;
  p.a.d_v = dims->d_v;
  p.a.d_c = dims->d_c;
  p.a.d_r = dims->d_r;
  p.a.t_max = dims->t_max;
  p.a.S = num_splits;
  p.a.split_rows = split_rows;
  p.a.scale_log2 = scale_log2(dims);
  p.a.fused = fused ? 1 : 0;
  p.a.block_table = block_table;
  p.a.page_rows = paging ? paging->page_rows : 0;
  p.a.max_pages = paging ? paging->max_pages : 0;
  p.a.n_pages = paging ? paging->n_pages : 0;
  fill_inv_freq(dims, p.inv_freq);
  hipStream_t s = static_cast<hipStream_t>(stream);

  if (dims->dtype == GVA_DTYPE_BF16) {
    if (dims->d_c % 32 != 0 || dims->d_c > 512 || dims->d_r % 8 != 0 || dims->d_r > 64)
      return GVA_ERR_UNSUPPORTED;
    // the fused prologue absorbs at least one 32-column chunk of the query
    if (fused && dims->d_c == 0) return GVA_ERR_UNSUPPORTED;
    const int nrc = (dims->d_r + 31) / 32;
    const int nw = fused && paging == nullptr ? decode_waves(n_items, device_cu_count()) : kWaves;
    DecodeFn fn = pick_bf16_decode(hpg, dims->d_v, nrc, fused, paging != nullptr, decode_kr_stream(dims), nw);
    if (fn == nullptr) return GVA_ERR_UNSUPPORTED;
    if (!launch) return GVA_OK;
    hipLaunchKernelGGL(fn, dim3((unsigned)n_items), dim3(64 * nw), 0, s, p);
  } else {
    if (paging != nullptr) return GVA_ERR_UNSUPPORTED;       // paged caches: bf16 only
    if (dims->d_v > kF32MaxDv || dims->d_c > 512 || dims->d_r > kF32MaxDr || hpg > kF32MaxHpg)
      return GVA_ERR_UNSUPPORTED;
    if (!launch) return GVA_OK;
    hipLaunchKernelGGL(decode_f32_kernel, dim3((unsigned)n_items), dim3(kThreads), 0, s, p);
  }
  return launch_status();
}

int combine_impl(const gva_dims* dims, const float* o_part, const float* lse_part, int32_t num_splits,
                 float* o, float* lse, void* stream, bool launch) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS) return GVA_ERR_INVALID_ARG;
  if (!o_part || !lse_part || !o) return GVA_ERR_INVALID_ARG;
  if (!aligned(o_part, 4) || !aligned(lse_part, 4) || !aligned(o, 4) || (lse && !aligned(lse, 4)))
    return GVA_ERR_INVALID_ARG;
  if (dims->d_v > kCombineMaxDv) return GVA_ERR_UNSUPPORTED;
  if (!launch) return GVA_OK;
  CombineParams p{};
  p.o_part = o_part;
  p.lse_part = lse_part;
  p.o = o;
  p.lse = lse;
  p.rows = dims->batch * dims->n_heads;
  p.S = num_splits;
  p.d_v = dims->d_v;
  const dim3 grid((p.rows + kWaves - 1) / kWaves);
  hipLaunchKernelGGL(combine_kernel, grid, dim3(kThreads), 0, static_cast<hipStream_t>(stream), p);
  return launch_status();
}

// ---------------------------------------------------------- whole step
// One decode step in one call: the absorption (inside the attention launch,
// or its own launch, as gva_prefer_fused decides), the attention, and the
// combine when there are several splits.  The intermediate buffers -- the
// absorbed queries of the separate path and the split partials -- live in
// a workspace; with one split the attention writes o and lse directly.
constexpr size_t kWorkspaceAlign = 256;

struct StepLayout {
  bool fused;
  size_t q_abs, q_rot, o_part, lse_part;   // byte offsets into the workspace
  size_t bytes;                            // workspace bytes the step uses
};

inline size_t ws_round(size_t x) { return (x + kWorkspaceAlign - 1) / kWorkspaceAlign * kWorkspaceAlign; }

int step_layout(const gva_dims* d, int32_t num_splits, int32_t split_rows, StepLayout& L) {
  const int st = check_dims(d);
  if (st != GVA_OK) return st;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS || split_rows < 0) return GVA_ERR_INVALID_ARG;
  L = StepLayout{};
  L.fused = gva_prefer_fused(d, num_splits, split_rows, 0) != 0;
  const size_t rows = (size_t)d->batch * (size_t)d->n_heads;
  size_t off = 0;
  if (!L.fused) {
    L.q_abs = off;
    off += ws_round(rows * (size_t)d->d_v * 4);
    L.q_rot = off;
    off += ws_round(rows * (size_t)d->d_r * 4);
  }
  if (num_splits > 1) {
    L.o_part = off;
    off += ws_round(rows * (size_t)num_splits * (size_t)d->d_v * 4);
    L.lse_part = off;
    off += ws_round(rows * (size_t)num_splits * 4);
  }
  L.bytes = off;
  return GVA_OK;
}

// The step's launches on workspace ws (L.bytes bytes, 256-byte aligned).
// Every launch is validated before the first is enqueued.
// With launch = false only the checks run.
int decode_step_impl(const gva_dims* dims, const void* q, const void* m, void* v_cache, void* kr_cache,
                     const int32_t* lens, const void* v_new, const void* kr_new, int32_t num_splits,
                     int32_t split_rows, char* ws, const StepLayout& L, float* o, float* lse, void* stream,
                     bool launch = true) {
  if (!q || !m || !o || !lse) return GVA_ERR_INVALID_ARG;
  const int S = num_splits;
  float* q_abs = L.fused ? nullptr : reinterpret_cast<float*>(ws + L.q_abs);
  float* q_rot = (L.fused || dims->d_r == 0) ? nullptr : reinterpret_cast<float*>(ws + L.q_rot);
  float* o_part = S > 1 ? reinterpret_cast<float*>(ws + L.o_part) : o;
  float* lse_part = S > 1 ? reinterpret_cast<float*>(ws + L.lse_part) : lse;
  const void* fq = L.fused ? q : nullptr;
  const void* fm = L.fused ? m : nullptr;
  for (int pass = 0; pass < (launch ? 2 : 1); ++pass) {   // pass 0 checks, pass 1 launches
    const bool go = pass == 1;
    int st = GVA_OK;
    if (!L.fused) st = absorb_impl(dims, 1, q, m, lens, q_abs, q_rot, stream, go);
    if (st == GVA_OK)
      st = decode_attention_impl(dims, nullptr, nullptr, fq, fm, q_abs, q_rot, v_cache, kr_cache, lens, v_new,
                                 kr_new, S, split_rows, o_part, lse_part, stream, go);
    if (st == GVA_OK && S > 1) st = combine_impl(dims, o_part, lse_part, S, o, lse, stream, go);
    if (st != GVA_OK) return st;
  }
  return GVA_OK;
}

}  // namespace

// ------------------------------------------------------- static scratch
// The workspace of gva_decode_step_static, for callers that cannot
// allocate: a file-scope device array, one copy on every GPU the library
// runs on, held until the process ends.  In host code `scratch` names a
// host-side stand-in, never the device memory: its device address is
// looked up once per device (hipGetSymbolAddress, with that device current)
// and only that address is passed to the kernels.
static __device__ __align__(256) unsigned char scratch[GVA_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_dev[kMaxDevices];   // per device: the address of its copy of scratch

int static_scratch(char** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return GVA_ERR_HIP;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (scratch_dev[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return GVA_ERR_HIP;
    scratch_dev[dev] = ptr;
  }
  *out = static_cast<char*>(scratch_dev[dev]);
  return GVA_OK;
}

}  // namespace

extern "C" {


int gva_version(void) { return 20000; }

const char* gva_status_string(int status) {
  switch (status) {
    case GVA_OK: return "ok";
    case GVA_ERR_INVALID_ARG: return "invalid argument";
    case GVA_ERR_UNSUPPORTED: return "unsupported shape";
    case GVA_ERR_HIP: return "HIP runtime error";
    case GVA_ERR_SCRATCH: return "the step needs more than the static scratch buffer (GVA_STATIC_SCRATCH_BYTES)";
  }
  return "unknown status";
}

int gva_append_kv(const gva_dims* dims, void* v_cache, void* kr_cache, const void* v_new,
                  const void* kr_new, const int32_t* seq, const int32_t* pos, int32_t n_rows,
                  void* stream) {
  return append_impl(dims, nullptr, nullptr, v_cache, kr_cache, v_new, kr_new, seq, pos, n_rows, stream);
}

int gva_absorb_query(const gva_dims* dims, const void* q, const void* m, const int32_t* lens,
                     float* q_abs, float* q_rot, void* stream) {
  return absorb_impl(dims, 1, q, m, lens, q_abs, q_rot, stream);
}


int gva_decode_attention(const gva_dims* dims, const void* q, const void* m, const float* q_abs,
                         const float* q_rot, void* v_cache, void* kr_cache,
                         const int32_t* lens, const void* v_new, const void* kr_new,
                         int32_t num_splits, int32_t split_rows, float* o_part, float* lse_part,
                         void* stream) {
  return decode_attention_impl(dims, nullptr, nullptr, q, m, q_abs, q_rot, v_cache, kr_cache, lens, v_new,
                               kr_new, num_splits, split_rows, o_part, lse_part, stream);
}

int gva_paged_decode_attention(const gva_dims* dims, const gva_paging* paging, const void* q, const void* m,
                               const float* q_abs, const float* q_rot, void* v_pool, void* kr_pool,
                               const int32_t* block_table, const int32_t* lens, const void* v_new,
                               const void* kr_new, int32_t num_splits, int32_t split_rows, float* o_part,
                               float* lse_part, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  st = check_paging(dims, paging, block_table);
  if (st != GVA_OK) return st;
  return decode_attention_impl(dims, paging, block_table, q, m, q_abs, q_rot, v_pool, kr_pool, lens, v_new,
                               kr_new, num_splits, split_rows, o_part, lse_part, stream);
}

int gva_paged_append_kv(const gva_dims* dims, const gva_paging* paging, void* v_pool, void* kr_pool,
                        const int32_t* block_table, const void* v_new, const void* kr_new, const int32_t* seq,
                        const int32_t* pos, int32_t n_rows, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  st = check_paging(dims, paging, block_table);
  if (st != GVA_OK) return st;
  return append_impl(dims, paging, block_table, v_pool, kr_pool, v_new, kr_new, seq, pos, n_rows, stream);
}

int gva_gqa_decode_attention(const gva_dims* dims, const void* q, int32_t q_stride,
                             const void* k_cache, const void* v_cache, const int32_t* lens,
                             int32_t num_splits, int32_t split_rows, float* o_part, float* lse_part,
                             void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS) return GVA_ERR_INVALID_ARG;
  if (split_rows < 0 || split_rows % kTileRows != 0) return GVA_ERR_INVALID_ARG;
  if (!q || !k_cache || !v_cache || !lens || !o_part || !lse_part) return GVA_ERR_INVALID_ARG;
  if (q_stride < dims->d_v) return GVA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(lens, 4) ||
      !aligned(o_part, 16) || !aligned(lse_part, 4))
    return GVA_ERR_INVALID_ARG;
  if (dims->dtype != GVA_DTYPE_BF16 || q_stride % 8 != 0) return GVA_ERR_UNSUPPORTED;
  if (dims->t_max % kLayoutRows != 0) return GVA_ERR_UNSUPPORTED;
  if ((double)dims->t_max * dims->d_v * 2.0 >= 2147483648.0 - 16777216.0) return GVA_ERR_UNSUPPORTED;
  const int hpg = dims->n_heads / dims->n_groups;
  const long long n_items = decode_grid(dims, num_splits, split_rows);
  if (n_items > 0x7FFFFFFFLL) return GVA_ERR_UNSUPPORTED;
  DecodeFn fn = pick_gqa_decode(hpg, dims->d_v);
  if (fn == nullptr) return GVA_ERR_UNSUPPORTED;

  DecodeParams p{};
  memset(&p, 0, sizeof(p));
  p.a.q = q;
  p.a.v = const_cast<void*>(v_cache);       // read only: the GQA kernel never appends
  p.a.k_gqa = k_cache;
  p.a.q_stride = q_stride;
  p.a.lens = lens;
  p.a.o_part = o_part;
  p.a.lse_part = lse_part;
  p.a.B = dims->batch;
  p.a.H = dims->n_heads;
  p.a.G = dims->n_groups;
  p.a.d_v = dims->d_v;
  p.a.d_c = dims->d_v;
  p.a.d_r = 0;
  p.a.t_max = dims->t_max;
  p.a.S = num_splits;
  p.a.split_rows = split_rows;
  const double sc = dims->scale > 0.0 ? dims->scale : 1.0 / sqrt((double)dims->d_v);
  p.a.scale_log2 = (float)(sc * kLog2e);
  hipLaunchKernelGGL(fn, dim3((unsigned)n_items), dim3(kThreads), 0, static_cast<hipStream_t>(stream), p);
  return launch_status();
}

int gva_prefill_absorb(const gva_dims* dims, int32_t n_new, const void* q, const void* m,
                       const int32_t* lens, float* q_abs, float* q_rot, void* stream) {
  if (dims != nullptr && (n_new < 1 || n_new > dims->t_max)) return GVA_ERR_INVALID_ARG;
  return absorb_impl(dims, n_new, q, m, lens, q_abs, q_rot, stream);
}

int gva_combine(const gva_dims* dims, const float* o_part, const float* lse_part, int32_t num_splits,
                float* o, float* lse, void* stream) {
  return combine_impl(dims, o_part, lse_part, num_splits, o, lse, stream, true);
}

int gva_decode_workspace_size(const gva_dims* dims, int32_t num_splits, int32_t split_rows, size_t* bytes) {
  if (bytes == nullptr) return GVA_ERR_INVALID_ARG;
  StepLayout L;
  const int st = step_layout(dims, num_splits, split_rows, L);
  if (st != GVA_OK) return st;
  *bytes = L.bytes;
  return GVA_OK;
}

int gva_decode_step(const gva_dims* dims, const void* q, const void* m, void* v_cache, void* kr_cache,
                    const int32_t* lens, const void* v_new, const void* kr_new, int32_t num_splits,
                    int32_t split_rows, void* workspace, size_t workspace_bytes, float* o, float* lse,
                    void* stream) {
  StepLayout L;
  const int st = step_layout(dims, num_splits, split_rows, L);
  if (st != GVA_OK) return st;
  if (L.bytes > 0 && (workspace == nullptr || workspace_bytes < L.bytes || !aligned(workspace, kWorkspaceAlign)))
    return GVA_ERR_INVALID_ARG;
  return decode_step_impl(dims, q, m, v_cache, kr_cache, lens, v_new, kr_new, num_splits, split_rows,
                          static_cast<char*>(workspace), L, o, lse, stream);
}

int gva_decode_step_static(const gva_dims* dims, const void* q, const void* m, void* v_cache, void* kr_cache,
                           const int32_t* lens, const void* v_new, const void* kr_new, int32_t num_splits,
                           int32_t split_rows, float* o, float* lse, void* stream) {
  StepLayout L;
  int st = step_layout(dims, num_splits, split_rows, L);
  if (st != GVA_OK) return st;
  if (L.bytes > (size_t)GVA_STATIC_SCRATCH_BYTES) return GVA_ERR_SCRATCH;
  // every check before the first runtime call (the checks see a stand-in
  // workspace address, aligned like the buffer, that nothing dereferences);
  // then the device's scratch
  char* const stand_in = reinterpret_cast<char*>(kWorkspaceAlign);
  st = decode_step_impl(dims, q, m, v_cache, kr_cache, lens, v_new, kr_new, num_splits, split_rows, stand_in, L, o,
                        lse, stream, false);
  if (st != GVA_OK) return st;
  char* ws = nullptr;
  if (L.bytes > 0) {
    st = static_scratch(&ws);
    if (st != GVA_OK) return st;
  }
  return decode_step_impl(dims, q, m, v_cache, kr_cache, lens, v_new, kr_new, num_splits, split_rows, ws, L, o, lse,
                          stream);
}

int gva_prefer_fused(const gva_dims* dims, int32_t num_splits, int32_t split_rows, int32_t n_cu) {
  if (check_dims(dims) != GVA_OK || num_splits < 1 || split_rows < 0) return 0;
  if (n_cu <= 0) n_cu = device_cu_count();
  if (decode_grid(dims, num_splits, split_rows) <= 2LL * n_cu) return 1;
  // bounded chunks: each workgroup streams up to split_rows value rows
  // against the (H/G) d_c map rows of its absorption
  const long long map_rows = (long long)(dims->n_heads / dims->n_groups) * dims->d_c;
  return split_rows > 0 && split_rows >= map_rows ? 1 : 0;
}

int gva_pick_splits(const gva_dims* dims, int32_t max_len, int64_t total_len, int32_t n_cu,
                    int32_t* split_rows) {
  if (split_rows != nullptr) *split_rows = 0;
  if (check_dims(dims) != GVA_OK) return 1;
  if (n_cu <= 0) n_cu = device_cu_count();
  if (max_len <= 0 || max_len > dims->t_max) max_len = dims->t_max;
  const long long streams = (long long)dims->batch * dims->n_groups;
  if (total_len <= 0) total_len = (long long)dims->batch * max_len;
  const long long row_bytes = (long long)dims->d_v * (long long)elem_size(dims);
  const bool spread = 2 * total_len < (long long)dims->batch * max_len;
  // Few streams (at most a quarter of the CUs): even splits, one workgroup
  // per CU, whatever the spread of the lengths (bounded chunks measured
  // 4-30% slower there).
  const bool few_streams = 4 * streams <= n_cu;
  if (spread && split_rows != nullptr && !few_streams) {
    // Ragged lengths: bounded chunks, so every workgroup streams about the
    // same bytes whatever its sequence's length.  Chunks with rows number
    // at most stream_rows / c + streams (ceil(L / c) < L / c + 1);
    // c is chosen so that they fit the kChunkItemsPerCu resident
    // workgroups per CU, one dispatch round with no tail, when the streams
    // leave room for that; none shorter than kMinChunkBytes of value rows,
    // nor than the (H/G) d_c map rows a chunk's fused absorption reads.
    const long long stream_rows = total_len * dims->n_groups;
    const long long slots = kChunkItemsPerCu * n_cu;
    const long long room = slots - streams > slots / 2 ? slots - streams : slots / 2;
    long long c = (stream_rows + room - 1) / room;
    long long min_rows = (kMinChunkBytes + row_bytes - 1) / row_bytes;
    const long long map_rows = (long long)(dims->n_heads / dims->n_groups) * dims->d_c;
    if (min_rows < map_rows) min_rows = map_rows;
    if (c < min_rows) c = min_rows;
    c = (c + kTileRows - 1) / kTileRows * kTileRows;
    long long s = (max_len + c - 1) / c;
    if (s > GVA_MAX_SPLITS) {
      c = ((max_len + GVA_MAX_SPLITS - 1) / GVA_MAX_SPLITS + kTileRows - 1) / kTileRows * kTileRows;
      s = (max_len + c - 1) / c;
    }
    if (s > 1) {
      *split_rows = (int32_t)c;
      return (int)s;
    }
  }
  // Even splits.  A workgroup streams its rows at the pace of its own chain
  // of memory round trips, so a launch of fewer workgroups than CUs is
  // bound by that chain, not by HBM; splitting the streams over more CUs
  // shortens it, but adds the combine launch and a prologue per split
  // (~3.5 us).  So: one split while a stream holds less than
  // kMinSplitStream bytes of value rows; else enough splits to give each
  // CU one workgroup (one resident workgroup per CU already streams close
  // to the HBM ceiling), none shorter than kMinSplitBytes, at most
  // kMaxEvenSplits (more partials cost the combine more than they save).
  long long s = 1;
  const long long stream_bytes = (long long)max_len * row_bytes;
  if (stream_bytes >= kMinSplitStream) {
    s = (n_cu + streams - 1) / streams;
    if (s > stream_bytes / kMinSplitBytes) s = stream_bytes / kMinSplitBytes;
    if (s > kMaxEvenSplits) s = kMaxEvenSplits;
  }
  // Lengths spread widely (mean below half the longest) over many streams:
  // the longest sequences set the tail, so cut them finer -- where they are
  // split at all (below kMinSplitStream the combine costs more than a split
  // saves).  Few streams already give each CU one workgroup.
  if (spread && s > 1 && !few_streams) s *= 2;
  if (s < 1) s = 1;
  if (s > GVA_MAX_SPLITS) s = GVA_MAX_SPLITS;
  return (int)s;
}

}  // extern "C"
