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
//   absorb_kernel        eq. absorb and the query rotation, standalone
//   decode_bf16_kernel   the hot path: fused absorb prologue, then a
//                        split-KV streaming loop over the value and
//                        positional-key rows of one (sequence, group, split)
//                        on the matrix cores, with an online softmax
//   decode_f32_kernel    fp32-storage variant on the vector ALUs
//   combine_kernel       log-sum-exp merge of the split partials
//
// Hot-loop design (bf16).  A workgroup owns one (b, g, split); its 4 waves
// take interleaved 32-row tiles.  Each lane loads 16-byte pieces of the V
// rows straight into MFMA operand registers (no LDS round trip), and every
// V tile serves all H/G heads of the group:
//   scores  S^T[t][n] = V[t][:] . Bq[:][n]           (v_mfma 16x16x32 bf16)
//           columns n hold each head's absorbed query twice, as a bf16 high
//           part and a bf16 low part (q~ = hi + lo to ~2^-16), mirrored so
//           a DPP mirror adds the pair; the positional key rides as one more
//           K-chunk of the same product
//   P.V     O^T[i][n] += V^T[i][t] P[t][n]            (v_mfma 16x16x32 bf16)
//           V^T comes from an identity-selector MFMA on the same registers,
//           P again split hi + lo, so both products keep ~fp32 accuracy
// The score layout the MFMA returns (lane = column, registers = 4 rows) is
// exactly the B-operand layout of the P.V product, so the softmax needs no
// cross-lane shuffles except the max over the four 16-lane rows.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "gva.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;             // waves per workgroup in the decode kernels
constexpr int kThreads = 64 * kWaves;
constexpr int kTileRows = 32;         // rows per tile = split granularity
constexpr int kMaxPairs = 32;         // d_r / 2 <= 32
constexpr float kLn2 = 0.693147180559945309417f;
constexpr double kLog2e = 1.44269504088896340736;

// ------------------------------------------------------------ parameters
struct AppendParams {
  void* v_cache;
  void* kr_cache;
  const void* v_new;
  const void* kr_new;
  const int32_t* seq;
  const int32_t* pos;
  int32_t B, G, t_max, d_v, d_r, n_rows;
  double inv_freq[kMaxPairs];
};

struct AbsorbParams {
  const void* q;
  const void* m;
  const int32_t* lens;
  float* q_abs;
  float* q_rot;
  int32_t B, H, d_v, d_c, d_r, t_max;
  double inv_freq[kMaxPairs];
};

struct DecodeParams {
  const void* q;          // fused path: raw query and maps
  const void* m;
  const float* q_abs;     // pre-absorbed path
  const float* q_rot;
  const void* v;
  const void* kr;
  const int32_t* lens;
  float* o_part;
  float* lse_part;
  int32_t B, H, G, d_v, d_c, d_r, t_max, S;
  float scale_log2;       // score scale * log2(e): softmax runs in base 2
  int32_t fused;
  double inv_freq[kMaxPairs];
};

struct CombineParams {
  const float* o_part;
  const float* lse_part;
  float* o;
  float* lse;
  int32_t rows, S, d_v;
};

// --------------------------------------------------------------- helpers
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_bits_to_f32(p[i]);
}

// Round a double to bfloat16 in one step: round to float with round-to-odd
// (truncate, then set the sticky bit if inexact), then nearest-even to bf16.
// Round-to-odd onto a format with >= 2 extra bits makes the second rounding
// exact-equivalent to a single rounding from the double.
__device__ __forceinline__ uint16_t f64_to_bf16_rne(double x) {
  if (x != x) return (uint16_t)0x7FC0;
  float f = (float)x;
  uint32_t u = __float_as_uint(f);
  double back = (double)f;
  if (back != x && !isinf(f)) {
    if (fabs(back) > fabs(x)) u -= 1;  // step the magnitude toward zero
    u |= 1u;
  }
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)(u >> 16);  // inf
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ void store_from_f64(T* p, int64_t i, double x);
template <>
__device__ __forceinline__ void store_from_f64<float>(float* p, int64_t i, double x) {
  p[i] = (float)x;
}
template <>
__device__ __forceinline__ void store_from_f64<uint16_t>(uint16_t* p, int64_t i, double x) {
  p[i] = f64_to_bf16_rne(x);
}

__device__ __forceinline__ int clamp_len(const int32_t* lens, int b, int t_max) {
  int L = lens[b];
  return L < 0 ? 0 : (L > t_max ? t_max : L);
}

// Split s of a sequence with L rows: [s*c, min(L, (s+1)*c)),
// c = kTileRows * ceil(ceil(L / S) / kTileRows).
__device__ __forceinline__ void split_rows(int L, int S, int s, int& r0, int& r1) {
  int per = (L + S - 1) / S;
  int chunk = ((per + kTileRows - 1) / kTileRows) * kTileRows;
  long long a = (long long)chunk * s, e = (long long)chunk * (s + 1);
  r0 = (int)(a < L ? a : L);
  r1 = (int)(e < L ? e : L);
}

// Workgroup index -> logical work item, XCD-aware.  The dispatcher deals
// consecutive workgroup ids round-robin over the 8 XCDs; this mapping gives
// each XCD one contiguous range of logical items, in order, so neighbouring
// items (the G groups of one (sequence, split), which read the same shared
// positional-key rows) run together on one XCD and share its L2.
__device__ __forceinline__ int xcd_remap(int x, int n) {
  const int per = n / 8, rem = n % 8;
  const int xcd = x % 8, slot = x / 8;
  return xcd * per + (xcd < rem ? xcd : rem) + slot;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// DPP control that pairs MFMA column n (a head's high part) with the column
// holding the same head's low part; columns are laid out
// [hi_0 .. hi_{P-1}, lo_{P-1} .. lo_0] so the pairing is a mirror.
template <int HPG>
struct Mirror;
template <> struct Mirror<1> { static constexpr int ctrl = 0xB1; };   // quad_perm [1,0,3,2]
template <> struct Mirror<2> { static constexpr int ctrl = 0x1B; };   // quad_perm [3,2,1,0]
template <> struct Mirror<4> { static constexpr int ctrl = 0x141; };  // row_half_mirror
template <> struct Mirror<8> { static constexpr int ctrl = 0x140; };  // row_mirror

template <int HPG>
__device__ __forceinline__ float mirror(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), Mirror<HPG>::ctrl, 0xF, 0xF, false));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 8 floats -> the bf16 high parts (RNE) or, with lo = true, the bf16 of the
// remainder x - hi.  hi + lo carries ~16 significant bits of x.
__device__ __forceinline__ bf16x8 split_hi_lo(const float* x, bool lo) {
  bf16x8 out;
#pragma unroll
  for (int j = 0; j < 8; j += 2) {
    f32x2 v = {x[j], x[j + 1]};
    bf16x2 h = __builtin_convertvector(v, bf16x2);
    if (lo) {
      f32x2 hv = __builtin_convertvector(h, f32x2);
      h = __builtin_convertvector(v - hv, bf16x2);
    }
    out[j] = h[0];
    out[j + 1] = h[1];
  }
  return out;
}

// ================================================================ append
template <typename T>
__global__ void __launch_bounds__(256) append_kernel(AppendParams p) {
  const int r = blockIdx.x;
  const int b = p.seq[r], ps = p.pos[r];
  if (b < 0 || b >= p.B || ps < 0 || ps >= p.t_max) return;
  const int tid = threadIdx.x;
  // value rows: 16-byte vectors (d_v * sizeof(T) is a multiple of 16)
  constexpr int kVec = 16 / sizeof(T);
  const int vec_per_row = p.d_v / kVec;
  const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const T*>(p.v_new) + (int64_t)r * p.G * p.d_v);
  for (int idx = tid; idx < p.G * vec_per_row; idx += blockDim.x) {
    const int g = idx / vec_per_row, c = idx % vec_per_row;
    T* dst = static_cast<T*>(p.v_cache) + (((int64_t)b * p.G + g) * p.t_max + ps) * p.d_v;
    reinterpret_cast<u32x4*>(dst)[c] = src[idx];
  }
  // positional key: rotate each pair at position ps in fp64 (eq. krope)
  const T* kin = static_cast<const T*>(p.kr_new) + (int64_t)r * p.d_r;
  T* kout = static_cast<T*>(p.kr_cache) + ((int64_t)b * p.t_max + ps) * p.d_r;
  for (int i = tid; i < p.d_r / 2; i += blockDim.x) {
    const double x0 = load_elem<T>(kin, 2 * i), x1 = load_elem<T>(kin, 2 * i + 1);
    const double a = (double)ps * p.inv_freq[i];
    const double c = cos(a), s = sin(a);
    store_from_f64<T>(kout, 2 * i, x0 * c - x1 * s);
    store_from_f64<T>(kout, 2 * i + 1, x0 * s + x1 * c);
  }
}

// ================================================================ absorb
template <typename T>
__global__ void __launch_bounds__(128) absorb_kernel(AbsorbParams p) {
  const int bh = blockIdx.x;
  const int b = bh / p.H, h = bh % p.H;
  const int W = p.d_c + p.d_r;
  const T* q = static_cast<const T*>(p.q) + (int64_t)bh * W;
  const T* m = static_cast<const T*>(p.m) + (int64_t)h * p.d_v * p.d_c;
  for (int i = threadIdx.x; i < p.d_v; i += blockDim.x) {
    float acc = 0.f;
    for (int k = 0; k < p.d_c; ++k) acc = fmaf(load_elem<T>(q, k), load_elem<T>(m, (int64_t)i * p.d_c + k), acc);
    p.q_abs[(int64_t)bh * p.d_v + i] = acc;
  }
  const int L = clamp_len(p.lens, b, p.t_max);
  const double pos = L > 0 ? (double)(L - 1) : 0.0;
  for (int i = threadIdx.x; i < p.d_r / 2; i += blockDim.x) {
    const double x0 = load_elem<T>(q, p.d_c + 2 * i), x1 = load_elem<T>(q, p.d_c + 2 * i + 1);
    const double a = pos * p.inv_freq[i];
    const double c = cos(a), s = sin(a);
    p.q_rot[(int64_t)bh * p.d_r + 2 * i] = (float)(x0 * c - x1 * s);
    p.q_rot[(int64_t)bh * p.d_r + 2 * i + 1] = (float)(x0 * s + x1 * c);
  }
}

// ========================================================= decode (bf16)
// HPG heads per group, DV value width, NRC = ceil(d_r / 32) positional
// K-chunks, DEPTH tiles of V held in registers (DEPTH-1 loads in flight).
template <int HPG, int DV, int NRC>
struct DecodeCfg {
  static constexpr int NC = DV / 32;                         // K-chunks per V row
  static constexpr int NB = DV / 16;                         // 16-wide i-blocks of the output
  static constexpr int DEPTH = DV >= 128 ? 3 : 4;
  static constexpr int QS_STRIDE = DV + 4;                   // padded LDS row (floats)
  static constexpr int QR_STRIDE = 32 * NRC + 4;
  static constexpr int LDS_PRO = HPG * (QS_STRIDE + QR_STRIDE);
  static constexpr int LDS_RED = kWaves * HPG * (DV + 2);
  static constexpr int LDS_FLOATS = LDS_PRO > LDS_RED ? LDS_PRO : LDS_RED;
};

template <int DV, int NRC>
struct Tile {
  bf16x8 v[2][DV / 32];                // [16-row half][K-chunk]
  bf16x8 k[2][NRC > 0 ? NRC : 1];      // positional key, [half][chunk]
};

template <int HPG, int DV, int NRC>
__global__ void __launch_bounds__(kThreads, 2) decode_bf16_kernel(DecodeParams p) {
  using Cfg = DecodeCfg<HPG, DV, NRC>;
  constexpr int NC = Cfg::NC, NB = Cfg::NB, DEPTH = Cfg::DEPTH;
  __shared__ float lds[Cfg::LDS_FLOATS];

  const int item = xcd_remap(blockIdx.x, gridDim.x);
  const int g = item % p.G;
  const int bs = item / p.G;
  const int s = bs % p.S;
  const int b = bs / p.S;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 15, qd = lane >> 4;     // MFMA column and 16-lane row
  const int h0 = g * HPG;
  const int L = clamp_len(p.lens, b, p.t_max);
  int r0, r1;
  split_rows(L, p.S, s, r0, r1);

  // ---- prologue: absorbed, rotated, scaled queries of the group's heads
  float* qs = lds;                                  // [HPG][QS_STRIDE]
  float* qr = lds + HPG * Cfg::QS_STRIDE;           // [HPG][QR_STRIDE]
  if (p.fused) {
    // q~_h = q^nope_h M_h^T on the matrix cores: A = M_h rows (i), K = d_c,
    // B = the query chunk broadcast to all 16 columns.
    const uint16_t* qg = static_cast<const uint16_t*>(p.q);
    const uint16_t* mg = static_cast<const uint16_t*>(p.m);
    const int W = p.d_c + p.d_r;
    for (int hl = w; hl < HPG; hl += kWaves) {
      const int h = h0 + hl;
      f32x4 acc[NB];
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) acc[ib] = f32x4{0.f, 0.f, 0.f, 0.f};
      const uint16_t* qrow = qg + ((int64_t)b * p.H + h) * W;
      const uint16_t* mh = mg + (int64_t)h * DV * p.d_c;
      for (int c = 0; c < p.d_c / 32; ++c) {
        const bf16x8 bq = as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + 32 * c + 8 * qd));
        bf16x8 am[NB];
#pragma unroll
        for (int ib = 0; ib < NB; ++ib)
          am[ib] = as_bf16x8(*reinterpret_cast<const u32x4*>(mh + (int64_t)(16 * ib + n) * p.d_c + 32 * c + 8 * qd));
#pragma unroll
        for (int ib = 0; ib < NB; ++ib) acc[ib] = mfma16(am[ib], bq, acc[ib]);
      }
      if (n == 0) {
#pragma unroll
        for (int ib = 0; ib < NB; ++ib)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) qs[hl * Cfg::QS_STRIDE + 16 * ib + 4 * qd + jj] = acc[ib][jj] * p.scale_log2;
      }
    }
    const int L1 = L > 0 ? L - 1 : 0;
    const int npair = p.d_r / 2;
    for (int idx = tid; idx < HPG * 16 * NRC; idx += kThreads) {
      const int hl = idx / (16 * NRC), i = idx % (16 * NRC);
      float y0 = 0.f, y1 = 0.f;
      if (i < npair) {
        const uint16_t* qrow = qg + ((int64_t)b * p.H + h0 + hl) * W + p.d_c;
        const double x0 = bf16_bits_to_f32(qrow[2 * i]), x1 = bf16_bits_to_f32(qrow[2 * i + 1]);
        const double a = (double)L1 * p.inv_freq[i];
        const double c = cos(a), sn = sin(a);
        y0 = (float)((x0 * c - x1 * sn) * (double)p.scale_log2);
        y1 = (float)((x0 * sn + x1 * c) * (double)p.scale_log2);
      }
      qr[hl * Cfg::QR_STRIDE + 2 * i] = y0;
      qr[hl * Cfg::QR_STRIDE + 2 * i + 1] = y1;
    }
  } else {
    for (int idx = tid; idx < HPG * DV; idx += kThreads) {
      const int hl = idx / DV, i = idx % DV;
      qs[hl * Cfg::QS_STRIDE + i] = p.q_abs[((int64_t)b * p.H + h0 + hl) * DV + i] * p.scale_log2;
    }
    for (int idx = tid; idx < HPG * 32 * NRC; idx += kThreads) {
      const int hl = idx / (32 * NRC), j = idx % (32 * NRC);
      qr[hl * Cfg::QR_STRIDE + j] =
          j < p.d_r ? p.q_rot[((int64_t)b * p.H + h0 + hl) * p.d_r + j] * p.scale_log2 : 0.f;
    }
  }
  __syncthreads();

  // Column roles: [hi_0 .. hi_{HPG-1}, lo_{HPG-1} .. lo_0, zero padding].
  const bool active = n < 2 * HPG;
  const bool is_lo = n >= HPG;
  const int col_head = !active ? 0 : (is_lo ? 2 * HPG - 1 - n : n);
  const bf16x8 zero8 = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
  bf16x8 bq[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const float* src = qs + col_head * Cfg::QS_STRIDE + 32 * c + 8 * qd;
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = src[j];
    bq[c] = active ? split_hi_lo(x, is_lo) : zero8;
  }
  bf16x8 bk[NRC > 0 ? NRC : 1];
#pragma unroll
  for (int rc = 0; rc < NRC; ++rc) {
    const float* src = qr + col_head * Cfg::QR_STRIDE + 32 * rc + 8 * qd;
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = src[j];
    bk[rc] = active ? split_hi_lo(x, is_lo) : zero8;
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
  const uint16_t* vbase = static_cast<const uint16_t*>(p.v) + ((int64_t)b * p.G + g) * p.t_max * DV;
  const uint16_t* kbase = static_cast<const uint16_t*>(p.kr) + (int64_t)b * p.t_max * p.d_r;
  const int kvec = p.d_r / 8;                      // 16-byte vectors per key row

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int ib = 0; ib < NB; ++ib) acc[ib] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int ntiles = (r1 - r0 + kTileRows - 1) / kTileRows;
  const int my_tiles = ntiles > w ? (ntiles - w + kWaves - 1) / kWaves : 0;

  auto tile_row = [&](int j) { return r0 + (w + kWaves * j) * kTileRows; };
  auto load_tile = [&](Tile<DV, NRC>& t, int row0) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      int row = row0 + 16 * hf + n;
      row = row < r1 ? row : r1 - 1;   // clamp: rows past the end are finite, masked later
      const u32x4* vr = reinterpret_cast<const u32x4*>(vbase + (int64_t)row * DV);
#pragma unroll
      for (int c = 0; c < NC; ++c) t.v[hf][c] = as_bf16x8(__builtin_nontemporal_load(vr + 4 * c + qd));
#pragma unroll
      for (int rc = 0; rc < NRC; ++rc) {
        int kv = 4 * rc + qd;
        kv = kv < kvec ? kv : kvec - 1;  // lanes past d_r reload a valid piece; its weight is 0
        t.k[hf][rc] = as_bf16x8(*(reinterpret_cast<const u32x4*>(kbase + (int64_t)row * p.d_r) + kv));
      }
    }
  };
  auto compute_tile = [&](const Tile<DV, NRC>& t, int row0) {
    // scores: rows 16*hf + 4*qd + jj of the tile, column n
    f32x4 sc[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      sc[hf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) sc[hf] = mfma16(t.v[hf][c], bq[c], sc[hf]);
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
    if (row0 + kTileRows > r1) {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (row0 + 16 * (k >> 2) + 4 * qd + (k & 3) >= r1) x[k] = -INFINITY;
    }
    float mt = x[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) mt = fmaxf(mt, x[k]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    if (__ballot(m_new > m_run) != 0) {
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

  Tile<DV, NRC> buf[DEPTH];
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d)
    if (d < my_tiles) load_tile(buf[d], tile_row(d));
  for (int jt = 0; jt < my_tiles; jt += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int j = jt + d;
      if (j < my_tiles) {
        const int jn = j + DEPTH - 1;
        if (jn < my_tiles) load_tile(buf[(d + DEPTH - 1) % DEPTH], tile_row(jn));
        compute_tile(buf[d], tile_row(j));
      }
    }
  }

  // ---- merge the waves and write this split's partial
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
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
  for (int idx = tid; idx < HPG * DV; idx += kThreads) {
    const int hl = idx / DV, i = idx % DV;
    float mx = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) mx = fmaxf(mx, red[(ww * HPG + hl) * RS]);
    float o = 0.f, lsum = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww) {
        const float* rec = red + (ww * HPG + hl) * RS;
        const float sc = rec[0] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(rec[0] - mx);
        lsum += rec[1] * sc;
        o += rec[2 + i] * sc;
      }
      o /= lsum;
    }
    const int64_t prow = ((int64_t)b * p.H + h0 + hl) * p.S + s;
    p.o_part[prow * DV + i] = o;
    if (i == 0) p.lse_part[prow] = mx == -INFINITY ? -INFINITY : (mx + log2f(lsum)) * kLn2;
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

  const int item = xcd_remap(blockIdx.x, gridDim.x);
  const int g = item % p.G;
  const int bs = item / p.G;
  const int s = bs % p.S;
  const int b = bs / p.S;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int hpg = p.H / p.G, h0 = g * hpg;
  const int DV = p.d_v, DR = p.d_r;
  const int L = clamp_len(p.lens, b, p.t_max);
  int r0, r1;
  split_rows(L, p.S, s, r0, r1);

  if (p.fused) {
    const float* qg = static_cast<const float*>(p.q);
    const float* mg = static_cast<const float*>(p.m);
    const int W = p.d_c + DR;
    for (int idx = tid; idx < hpg * DV; idx += kThreads) {
      const int hl = idx / DV, i = idx % DV;
      const float* qrow = qg + ((int64_t)b * p.H + h0 + hl) * W;
      const float* mrow = mg + ((int64_t)(h0 + hl) * DV + i) * p.d_c;
      float a = 0.f;
      for (int k = 0; k < p.d_c; ++k) a = fmaf(qrow[k], mrow[k], a);
      qs[hl][i] = a * p.scale_log2;
    }
    const int L1 = L > 0 ? L - 1 : 0;
    for (int idx = tid; idx < hpg * (DR / 2); idx += kThreads) {
      const int hl = idx / (DR / 2), i = idx % (DR / 2);
      const float* qrow = qg + ((int64_t)b * p.H + h0 + hl) * W + p.d_c;
      const double x0 = qrow[2 * i], x1 = qrow[2 * i + 1];
      const double a = (double)L1 * p.inv_freq[i];
      const double c = cos(a), sn = sin(a);
      qr[hl][2 * i] = (float)((x0 * c - x1 * sn) * (double)p.scale_log2);
      qr[hl][2 * i + 1] = (float)((x0 * sn + x1 * c) * (double)p.scale_log2);
    }
  } else {
    for (int idx = tid; idx < hpg * DV; idx += kThreads) {
      const int hl = idx / DV, i = idx % DV;
      qs[hl][i] = p.q_abs[((int64_t)b * p.H + h0 + hl) * DV + i] * p.scale_log2;
    }
    for (int idx = tid; idx < hpg * DR; idx += kThreads) {
      const int hl = idx / DR, j = idx % DR;
      qr[hl][j] = p.q_rot[((int64_t)b * p.H + h0 + hl) * DR + j] * p.scale_log2;
    }
  }
  __syncthreads();

  const float* vb = static_cast<const float*>(p.v) + ((int64_t)b * p.G + g) * p.t_max * DV;
  const float* kb = static_cast<const float*>(p.kr) + (int64_t)b * p.t_max * DR;
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
        const float* vr = vb + (int64_t)t * DV;
        for (int i = 0; i < DV; ++i) {
          const float v = vr[i];
#pragma unroll
          for (int h = 0; h < kF32MaxHpg; ++h)
            if (h < hpg) sc[h] = fmaf(qs[h][i], v, sc[h]);
        }
        const float* kr = kb + (int64_t)t * DR;
        for (int j = 0; j < DR; ++j) {
          const float k = kr[j];
#pragma unroll
          for (int h = 0; h < kF32MaxHpg; ++h)
            if (h < hpg) sc[h] = fmaf(qr[h][j], k, sc[h]);
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
      for (int t = 0; t < nrow; ++t) {
        const float* vr = vb + (int64_t)(row0 + t) * DV;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = lane + 64 * u;
          if (i < DV) {
            const float v = vr[i];
#pragma unroll
            for (int h = 0; h < kF32MaxHpg; ++h)
              if (h < hpg) acc[h][u] = fmaf(pb[w][t][h], v, acc[h][u]);
          }
        }
      }
    }
    __syncthreads();
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
    const int64_t prow = ((int64_t)b * p.H + h0 + hl) * p.S + s;
    p.o_part[prow * DV + i] = o;
    if (i == 0) p.lse_part[prow] = mx == -INFINITY ? -INFINITY : (mx + log2f(lsum)) * kLn2;
  }
}

// =============================================================== combine
__global__ void __launch_bounds__(128) combine_kernel(CombineParams p) {
  __shared__ float wts[GVA_MAX_SPLITS];
  __shared__ float lse_row;
  const int row = blockIdx.x;
  const float* lp = p.lse_part + (int64_t)row * p.S;
  if (threadIdx.x == 0) {
    float mx = -INFINITY;
    for (int s = 0; s < p.S; ++s) mx = fmaxf(mx, lp[s]);
    float z = 0.f;
    if (mx != -INFINITY)
      for (int s = 0; s < p.S; ++s)
        if (lp[s] != -INFINITY) z += expf(lp[s] - mx);
    lse_row = mx == -INFINITY ? -INFINITY : mx + logf(z);
  }
  __syncthreads();
  const float big = lse_row;
  for (int s = threadIdx.x; s < p.S; s += blockDim.x)
    wts[s] = (big == -INFINITY || lp[s] == -INFINITY) ? 0.f : expf(lp[s] - big);
  __syncthreads();
  const float* op = p.o_part + (int64_t)row * p.S * p.d_v;
  for (int i = threadIdx.x; i < p.d_v; i += blockDim.x) {
    float o = 0.f;
    for (int s = 0; s < p.S; ++s)
      if (wts[s] != 0.f) o = fmaf(wts[s], op[(int64_t)s * p.d_v + i], o);
    p.o[(int64_t)row * p.d_v + i] = o;
  }
  if (p.lse != nullptr && threadIdx.x == 0) p.lse[row] = big;
}

// ================================================================== host
bool aligned(const void* ptr, size_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

int check_dims(const gva_dims* d) {
  if (d == nullptr) return GVA_ERR_INVALID_ARG;
  if (d->batch < 1 || d->n_heads < 1 || d->n_groups < 1 || d->t_max < 1) return GVA_ERR_INVALID_ARG;
  if (d->n_heads % d->n_groups != 0) return GVA_ERR_INVALID_ARG;
  if (d->d_v < 1 || d->d_c < 0 || d->d_r < 0 || (d->d_r & 1)) return GVA_ERR_INVALID_ARG;
  if (d->dtype != GVA_DTYPE_F32 && d->dtype != GVA_DTYPE_BF16) return GVA_ERR_INVALID_ARG;
  if (!(d->scale >= 0.0) || !isfinite(d->scale)) return GVA_ERR_INVALID_ARG;
  if (d->d_r > 0 && (!(d->rope_base > 0.0) || !isfinite(d->rope_base))) return GVA_ERR_INVALID_ARG;
  if (d->d_c + d->d_r < 1) return GVA_ERR_INVALID_ARG;
  if (d->d_r / 2 > kMaxPairs) return GVA_ERR_UNSUPPORTED;
  return GVA_OK;
}

size_t elem_size(const gva_dims* d) { return d->dtype == GVA_DTYPE_BF16 ? 2 : 4; }

void fill_inv_freq(const gva_dims* d, double* out) {
  for (int i = 0; i < kMaxPairs; ++i)
    out[i] = (i < d->d_r / 2) ? pow(d->rope_base, -2.0 * (double)i / (double)d->d_r) : 0.0;
}

float scale_log2(const gva_dims* d) {
  const double sc = d->scale > 0.0 ? d->scale : 1.0 / sqrt((double)(d->d_c + d->d_r));
  return (float)(sc * kLog2e);
}

int launch_status() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? GVA_OK : GVA_ERR_HIP;
}

using DecodeFn = void (*)(DecodeParams);

template <int HPG, int DV>
DecodeFn pick_nrc(int nrc) {
  switch (nrc) {
    case 0: return decode_bf16_kernel<HPG, DV, 0>;
    case 1: return decode_bf16_kernel<HPG, DV, 1>;
    case 2: return decode_bf16_kernel<HPG, DV, 2>;
  }
  return nullptr;
}

template <int HPG>
DecodeFn pick_dv(int dv, int nrc) {
  switch (dv) {
    case 64: return pick_nrc<HPG, 64>(nrc);
    case 128: return pick_nrc<HPG, 128>(nrc);
  }
  return nullptr;
}

DecodeFn pick_bf16_decode(int hpg, int dv, int nrc) {
  switch (hpg) {
    case 1: return pick_dv<1>(dv, nrc);
    case 2: return pick_dv<2>(dv, nrc);
    case 4: return pick_dv<4>(dv, nrc);
    case 8: return pick_dv<8>(dv, nrc);
  }
  return nullptr;
}

}  // namespace

extern "C" {

int gva_version(void) { return 10000; }

const char* gva_status_string(int status) {
  switch (status) {
    case GVA_OK: return "ok";
    case GVA_ERR_INVALID_ARG: return "invalid argument";
    case GVA_ERR_UNSUPPORTED: return "unsupported shape";
    case GVA_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

int gva_append_kv(const gva_dims* dims, void* v_cache, void* kr_cache, const void* v_new,
                  const void* kr_new, const int32_t* seq, const int32_t* pos, int32_t n_rows,
                  void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (n_rows < 0) return GVA_ERR_INVALID_ARG;
  if (n_rows == 0) return GVA_OK;
  if (!v_cache || !v_new || !seq || !pos) return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && (!kr_cache || !kr_new)) return GVA_ERR_INVALID_ARG;
  if (!aligned(v_cache, 16) || !aligned(v_new, 16) || !aligned(seq, 4) || !aligned(pos, 4))
    return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && (!aligned(kr_cache, 4) || !aligned(kr_new, 4))) return GVA_ERR_INVALID_ARG;
  if ((dims->d_v * elem_size(dims)) % 16 != 0) return GVA_ERR_UNSUPPORTED;
  AppendParams p;
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
  fill_inv_freq(dims, p.inv_freq);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dims->dtype == GVA_DTYPE_BF16)
    hipLaunchKernelGGL(append_kernel<uint16_t>, dim3(n_rows), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(append_kernel<float>, dim3(n_rows), dim3(256), 0, s, p);
  return launch_status();
}

int gva_absorb_query(const gva_dims* dims, const void* q, const void* m, const int32_t* lens,
                     float* q_abs, float* q_rot, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (!q || !m || !lens || !q_abs) return GVA_ERR_INVALID_ARG;
  if (dims->d_r > 0 && !q_rot) return GVA_ERR_INVALID_ARG;
  if (!aligned(q, elem_size(dims)) || !aligned(m, elem_size(dims)) || !aligned(lens, 4) ||
      !aligned(q_abs, 4) || (q_rot && !aligned(q_rot, 4)))
    return GVA_ERR_INVALID_ARG;
  AbsorbParams p;
  p.q = q;
  p.m = m;
  p.lens = lens;
  p.q_abs = q_abs;
  p.q_rot = q_rot;
  p.B = dims->batch;
  p.H = dims->n_heads;
  p.d_v = dims->d_v;
  p.d_c = dims->d_c;
  p.d_r = dims->d_r;
  p.t_max = dims->t_max;
  fill_inv_freq(dims, p.inv_freq);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(dims->batch * dims->n_heads);
  if (dims->dtype == GVA_DTYPE_BF16)
    hipLaunchKernelGGL(absorb_kernel<uint16_t>, grid, dim3(128), 0, s, p);
  else
    hipLaunchKernelGGL(absorb_kernel<float>, grid, dim3(128), 0, s, p);
  return launch_status();
}

int gva_decode_attention(const gva_dims* dims, const void* q, const void* m, const float* q_abs,
                         const float* q_rot, const void* v_cache, const void* kr_cache,
                         const int32_t* lens, int32_t num_splits, float* o_part, float* lse_part,
                         void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS) return GVA_ERR_INVALID_ARG;
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

  const int hpg = dims->n_heads / dims->n_groups;
  const long long n_items = (long long)dims->batch * dims->n_groups * num_splits;
  if (n_items > 0x7FFFFFFFLL) return GVA_ERR_UNSUPPORTED;

  DecodeParams p;
  p.q = q;
  p.m = m;
  p.q_abs = q_abs;
  p.q_rot = q_rot;
  p.v = v_cache;
  p.kr = kr_cache;
  p.lens = lens;
  p.o_part = o_part;
  p.lse_part = lse_part;
  p.B = dims->batch;
  p.H = dims->n_heads;
  p.G = dims->n_groups;
  p.d_v = dims->d_v;
  p.d_c = dims->d_c;
  p.d_r = dims->d_r;
  p.t_max = dims->t_max;
  p.S = num_splits;
  p.scale_log2 = scale_log2(dims);
  p.fused = fused ? 1 : 0;
  fill_inv_freq(dims, p.inv_freq);
  hipStream_t s = static_cast<hipStream_t>(stream);

  if (dims->dtype == GVA_DTYPE_BF16) {
    if (dims->d_c % 32 != 0 || dims->d_c > 512 || dims->d_r % 8 != 0 || dims->d_r > 64)
      return GVA_ERR_UNSUPPORTED;
    const int nrc = (dims->d_r + 31) / 32;
    DecodeFn fn = pick_bf16_decode(hpg, dims->d_v, nrc);
    if (fn == nullptr) return GVA_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(fn, dim3((unsigned)n_items), dim3(kThreads), 0, s, p);
  } else {
    if (dims->d_v > kF32MaxDv || dims->d_c > 512 || dims->d_r > kF32MaxDr || hpg > kF32MaxHpg)
      return GVA_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(decode_f32_kernel, dim3((unsigned)n_items), dim3(kThreads), 0, s, p);
  }
  return launch_status();
}

int gva_combine(const gva_dims* dims, const float* o_part, const float* lse_part, int32_t num_splits,
                float* o, float* lse, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS) return GVA_ERR_INVALID_ARG;
  if (!o_part || !lse_part || !o) return GVA_ERR_INVALID_ARG;
  if (!aligned(o_part, 4) || !aligned(lse_part, 4) || !aligned(o, 4) || (lse && !aligned(lse, 4)))
    return GVA_ERR_INVALID_ARG;
  CombineParams p;
  p.o_part = o_part;
  p.lse_part = lse_part;
  p.o = o;
  p.lse = lse;
  p.rows = dims->batch * dims->n_heads;
  p.S = num_splits;
  p.d_v = dims->d_v;
  hipLaunchKernelGGL(combine_kernel, dim3(p.rows), dim3(128), 0, static_cast<hipStream_t>(stream), p);
  return launch_status();
}

int gva_pick_splits(const gva_dims* dims, int32_t max_len, int32_t n_cu) {
  if (check_dims(dims) != GVA_OK) return 1;
  if (n_cu <= 0) {
    int dev = 0, cu = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cu > 0)
      n_cu = cu;
    else
      n_cu = 256;
  }
  if (max_len <= 0) max_len = dims->t_max;
  const long long streams = (long long)dims->batch * dims->n_groups;
  // aim for ~4 resident workgroups per CU, but keep each split >= 256 rows
  long long s = (4LL * n_cu + streams - 1) / streams;
  const long long max_by_len = (max_len + 255) / 256;
  if (s > max_by_len) s = max_by_len;
  if (s < 1) s = 1;
  if (s > GVA_MAX_SPLITS) s = GVA_MAX_SPLITS;
  return (int)s;
}

}  // extern "C"
