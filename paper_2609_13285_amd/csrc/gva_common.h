// Shared by the GVA kernel sources: constants, parameter blocks, device
// helpers and the host-side argument checks.  Everything here has internal
// linkage (anonymous namespace, inline), so each source compiles its own copy.

#pragma once

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
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;             // waves per workgroup in the decode kernels
constexpr int kThreads = 64 * kWaves;
constexpr int kTileRows = 32;         // rows per compute tile = split granularity
constexpr int kLayoutRows = 16;       // rows per cache layout tile
constexpr int kMaxPairs = 32;         // d_r / 2 <= 32
constexpr float kLn2 = 0.693147180559945309417f;
constexpr double kLog2e = 1.44269504088896340736;
constexpr int kBufferWord3 = 0x00020000;   // raw buffer descriptor, 32-bit data format
constexpr int kAuxNT = 2;                  // non-temporal: the V stream is read once
constexpr int kMaxPages = 4096;            // paged caches: block-table entries per sequence

// ------------------------------------------------------------ parameters
struct AppendParams {
  void* v_cache;
  void* kr_cache;
  const void* v_new;
  const void* kr_new;
  const int32_t* seq;
  const int32_t* pos;
  int32_t B, G, t_max, d_v, d_r, n_rows;
  const int32_t* block_table;   // paged caches (NULL: contiguous streams)
  int32_t page_rows, max_pages, n_pages;
  double inv_freq[kMaxPairs];
};

struct AbsorbParams {
  const void* q;
  const void* m;
  const int32_t* lens;
  float* q_abs;
  float* q_rot;
  int32_t B, H, d_v, d_c, d_r, t_max;   // B = query rows (sequences x n_per_seq)
  int32_t n_per_seq;                    // query rows per sequence: its last cached rows
  int32_t row_blocks;                   // bf16 kernel: 16-row blocks per workgroup (1..4)
  double inv_freq[kMaxPairs];
};

struct DecodeArgs {
  const void* q;          // fused path: raw query and maps
  const void* m;
  const float* q_abs;     // pre-absorbed path
  const float* q_rot;
  void* v;                                 // caches: read, and row L-1 written when pending
  void* kr;
  const int32_t* lens;
  float* o_part;
  float* lse_part;
  const void* v_new;      // optional: the current token's rows, used in place
  const void* kr_new;     // of cache row len-1 (see gva_decode_attention)
  const void* k_gqa;      // matched-GQA baseline: explicit key cache (tiled like v)
  int32_t q_stride;       // matched-GQA baseline: elements per query row
  int32_t B, H, G, d_v, d_c, d_r, t_max, S;
  int32_t split_rows;     // fixed rows per split (0: the even rule)
  float scale_log2;       // score scale * log2(e): softmax runs in base 2
  int32_t fused;
  const int32_t* block_table;   // paged caches: [B][max_pages] page ids
  int32_t page_rows, max_pages, n_pages;
};

struct DecodeParams {
  DecodeArgs a;           // scalars and pointers: read into registers at once
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
// equivalent to a single rounding from the double.
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

// Element offset of (t, i) inside one stream of the tiled cache layout.
template <typename T>
__host__ __device__ __forceinline__ int64_t tiled_off(int64_t t, int i, int D) {
  constexpr int P = 16 / (int)sizeof(T);
  return (t / kLayoutRows) * kLayoutRows * D + ((int64_t)(i / P) * kLayoutRows + t % kLayoutRows) * P + i % P;
}

__device__ __forceinline__ int clamp_len(const int32_t* lens, int b, int t_max) {
  int L = lens[b];
  return L < 0 ? 0 : (L > t_max ? t_max : L);
}

// Splits of a sequence with L rows: the first n of its S splits hold its
// rows, evenly: split s covers [s*k, min(L, (s+1)*k)) with
// k = kTileRows * ceil(ceil(L / n) / kTileRows), and splits from n on are
// empty.  Even splits (split_rows = 0): n = S.  Bounded chunks (split_rows
// = c > 0, a multiple of kTileRows): n = ceil(L / c), at least 1 and at
// most S, so every split holds at most c rows (unless S splits of c rows
// cannot cover L) and the splits of one sequence are equal.
__device__ __forceinline__ int split_count(int L, int S, int c) {
  if (c <= 0) return S;
  const int n = (L + c - 1) / c;
  return n < 1 ? 1 : (n > S ? S : n);
}

__device__ __forceinline__ void split_rows(int L, int S, int c, int s, int& r0, int& r1) {
  const int n = split_count(L, S, c);
  const int per = (L + n - 1) / n;
  const long long k = (long long)((per + kTileRows - 1) / kTileRows) * kTileRows;
  const long long a = k * s, e = k * (s + 1);
  r0 = (int)(a < L ? a : L);
  r1 = (int)(e < L ? e : L);
}

// Workgroup index -> logical work item, XCD-aware.  The dispatcher deals
// consecutive workgroup ids round-robin over the 8 XCDs; this mapping gives
// each XCD one contiguous range of logical items, in order.
__device__ __forceinline__ int xcd_remap(int x, int n) {
  const int per = n / 8, rem = n % 8;
  const int xcd = x % 8, slot = x / 8;
  return xcd * per + (xcd < rem ? xcd : rem) + slot;
}

// Workgroup -> (sequence b, split s, group g).  Each XCD reaches HBM
// through its own share of the fabric, so a launch takes as long as its
// busiest XCD: every XCD must get the same bytes.  The G groups of one
// (b, s) slot always land on one XCD, next to each other, and share the
// slot's positional-key rows in its L2.
//  - Even splits: the slots in split-major order (k = s B + b), each XCD
//    one contiguous range of them (xcd_remap), B * S * G workgroups.  An
//    XCD then holds the same splits of consecutive sequences: with S a
//    multiple of 8, split x of every sequence on XCD x, the same share of
//    each sequence whatever the lengths; with S = 1, whole sequences that
//    lie next to each other in memory.
//  - Bounded chunks (see chunk_item): the (b, s) slots in the order
//    chunks with rows, then empty slots, dealt round-robin over the XCDs
//    (slot k to XCD k mod 8), so chunks of every length spread over all of
//    them; the grid is B * S rounded up to 8, times G, and workgroups past
//    B * S are padding and return false.
// Every scalar argument the decode prologue needs, requested here in one
// round trip: left to itself the compiler fetches them where first used,
// several dependent kernel-argument round trips deep.  The memory clobber
// keeps the loads that follow after this point.
template <bool RAW_QUERY>
__device__ __forceinline__ void request_args(const DecodeArgs& a) {
  asm volatile("" ::"s"(a.B), "s"(a.H), "s"(a.G), "s"(a.S), "s"(a.t_max), "s"(a.split_rows), "s"(a.d_r),
               "s"(a.d_c), "s"(a.lens), "s"(a.v_new), "s"(a.kr_new),
               "s"(RAW_QUERY ? static_cast<const void*>(a.q) : static_cast<const void*>(a.q_abs)),
               "s"(RAW_QUERY ? a.m : static_cast<const void*>(a.q_rot)), "s"(gridDim.x)
               : "memory");
}

// Bounded chunks: the splits of sequence bb that hold rows (0 past the
// batch and for an empty sequence).
__device__ __forceinline__ int chunk_count(const DecodeArgs& p, int bb) {
  int L = bb < p.B ? p.lens[bb] : 0;
  L = L < 0 ? 0 : (L > p.t_max ? p.t_max : L);
  return L > 0 ? split_count(L, p.S, p.split_rows) : 0;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

// Bounded chunks: slot i of the B * S (sequence, split) slots.  Slots are
// numbered splits with rows first (sequence-major), then the empty splits,
// so the dispatcher hands out every chunk with rows before any workgroup
// that only records an empty split.  The map is a bijection of [0, B S)
// onto the slots, found by every wave of the workgroup from the lengths in
// two levels: lane l first sums the counts of the k = ceil(B / 64)
// sequences [l k, l k + k) (independent loads), a scan over the lanes
// finds the block holding slot i, and for k > 1 a second scan over that
// block's sequences (64 at a time) finds the sequence.  empty: the slot
// has no rows.
__device__ __forceinline__ void chunk_item(const DecodeArgs& p, int i, int& b, int& s, bool& empty) {
  const int lane = threadIdx.x & 63;
  const int k = (p.B + 63) >> 6;
  int n_sum = 0, nb = 0;
#pragma unroll 4
  for (int j = 0; j < k; ++j) {
    n_sum += chunk_count(p, lane * k + j);
    nb += lane * k + j < p.B ? 1 : 0;
  }
  const int F = wave_sum_int(n_sum);
  const bool full = i < F;                     // a split with rows
  const int kk = full ? i : i - F;
  // slots of the category per sequence: its splits with rows, or the rest
  auto pick = [&](int n, int valid) { return full ? n : valid * p.S - n; };
  const int cnt1 = pick(n_sum, nb);
  const int incl1 = wave_incl_scan(cnt1);
  const int j1 = min(__popcll(__ballot(incl1 <= kk)), 63);   // < 64 whenever i < B S
  int base = __shfl(incl1 - cnt1, j1, 64);
  // the slot's split within its sequence: the local-th with rows, or the
  // local-th empty one after those
  auto split_of = [&](int n, int local) { return full ? local : n + local; };
  b = 0;
  s = 0;
  if (k == 1) {                                // one sequence per lane: found
    b = __builtin_amdgcn_readfirstlane(j1);
    s = __builtin_amdgcn_readfirstlane(split_of(__shfl(n_sum, j1, 64), kk - base));
  } else {
    const int first = j1 * k;
    for (int c = 0; c < k; c += 64) {
      const int bb = first + c + lane;
      const bool in_blk = c + lane < k && bb < p.B;
      const int n = chunk_count(p, in_blk ? bb : p.B);
      const int cnt = in_blk ? pick(n, 1) : 0;
      const int incl = base + wave_incl_scan(cnt);
      const int j = __popcll(__ballot(incl <= kk));
      if (j < 64) {
        const int excl = __shfl(incl - cnt, j, 64);
        b = __builtin_amdgcn_readfirstlane(first + c + j);
        s = __builtin_amdgcn_readfirstlane(split_of(__shfl(n, j, 64), kk - excl));
        break;
      }
      base = __shfl(incl, 63, 64);
    }
  }
  empty = !full;
}

__device__ __forceinline__ bool work_item(const DecodeArgs& p, int& b, int& s, int& g, bool& empty) {
  const int x = blockIdx.x;
  empty = false;
  if (p.split_rows > 0) {
    const int slot = x >> 3;                   // the workgroup's place on its XCD (x mod 8)
    g = slot % p.G;
    const int i = 8 * (slot / p.G) + (x & 7);
    if (i >= p.B * p.S) return false;
    chunk_item(p, i, b, s, empty);
    return true;
  }
  const int item = xcd_remap(x, gridDim.x);
  g = item % p.G;
  const int k = item / p.G;
  s = k / p.B;
  b = k % p.B;
  return true;
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

// max of x over the four 16-lane rows of a wave (lanes l, l^16, l^32, l^48),
// with the gfx950 row-swap permutes (no LDS round trip)
__device__ __forceinline__ float max_over_rows(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum_over_rows(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
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

// dot product of eight bf16 pairs (two 16-byte pieces), fp32 accumulation.
// The pairs are taken with shufflevector: a bit_cast of one 32-bit element
// of the u32x4 compiled to four uses of element 0.
__device__ __forceinline__ float dot8_bf16(u32x4 x, u32x4 y) {
  const bf16x8 xv = as_bf16x8(x), yv = as_bf16x8(y);
  float acc = 0.f;
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(xv, xv, 0, 1), __builtin_shufflevector(yv, yv, 0, 1),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(xv, xv, 2, 3), __builtin_shufflevector(yv, yv, 2, 3),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(xv, xv, 4, 5), __builtin_shufflevector(yv, yv, 4, 5),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(xv, xv, 6, 7), __builtin_shufflevector(yv, yv, 6, 7),
                                        acc, false);
  return acc;
}

template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// sum over each aligned group of 16 lanes, every lane of the group receiving
// it: quad_perm [1,0,3,2], quad_perm [3,2,1,0], row_half_mirror, row_mirror
__device__ __forceinline__ float sum16(float x) {
  return dpp_add<0x140>(dpp_add<0x141>(dpp_add<0x1B>(dpp_add<0xB1>(x))));
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// 8 floats -> fp16 (RNE)
__device__ __forceinline__ f16x8 to_f16x8(const float* x) {
  f16x8 out;
#pragma unroll
  for (int j = 0; j < 8; j += 2) {
    const f16x2 h = __builtin_convertvector((f32x2{x[j], x[j + 1]}), f16x2);
    out[j] = h[0];
    out[j + 1] = h[1];
  }
  return out;
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

// cos/sin of an fp64 angle, evaluated in fp32 after an exact reduction by
// multiples of 2 pi in fp64 (Cody-Waite with 2 pi split into two doubles;
// each fma subtracts an exactly formed product).  Accurate to fp32 rounding
// for |a| < 2^40, which covers every position times a RoPE frequency <= 1.
__device__ __forceinline__ void sincos_reduced(double a, float& s, float& c) {
  constexpr double kInv2Pi = 0.15915494309189533577;
  constexpr double k2PiHi = 6.28318530717958623200;    // 2 pi rounded to double
  constexpr double k2PiLo = 2.44929359829470635445e-16; // 2 pi - k2PiHi
  const double k = rint(a * kInv2Pi);
  double r = fma(-k, k2PiHi, a);
  r = fma(-k, k2PiLo, r);
  sincosf((float)r, &s, &c);
}

// The query's positional slice, rotated at position pos and scaled: fp32 is
// all the score needs.
__device__ __forceinline__ void rotate_query_pair(float x0, float x1, double a, float scale, float& y0, float& y1) {
  float s, c;
  sincos_reduced(a, s, c);
  y0 = (x0 * c - x1 * s) * scale;
  y1 = (x0 * s + x1 * c) * scale;
}

__device__ __forceinline__ void rotate_pair(double x0, double x1, double a, double& y0, double& y1) {
  double s, c;
  sincos(a, &s, &c);
  y0 = x0 * c - x1 * s;
  y1 = x0 * s + x1 * c;
}

template <int DV, int NRC, bool GQA>
struct Tile {
  bf16x8 v[2][DV / 32];                // [16-row half][K-chunk]
  bf16x8 k[2][NRC > 0 ? NRC : 1];      // positional key, [half][chunk]
  bf16x8 kc[2][GQA ? DV / 32 : 1];     // matched-GQA baseline: explicit key rows
};

// ================================================================== host
inline bool aligned(const void* ptr, size_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

inline int check_dims(const gva_dims* d) {
  if (d == nullptr) return GVA_ERR_INVALID_ARG;
  if (d->batch < 1 || d->n_heads < 1 || d->n_groups < 1 || d->t_max < 1) return GVA_ERR_INVALID_ARG;
  if (d->n_heads % d->n_groups != 0) return GVA_ERR_INVALID_ARG;
  if (d->d_v < 1 || d->d_c < 0 || d->d_r < 0 || (d->d_r & 1)) return GVA_ERR_INVALID_ARG;
  if (d->dtype != GVA_DTYPE_F32 && d->dtype != GVA_DTYPE_BF16) return GVA_ERR_INVALID_ARG;
  if (!(d->scale >= 0.0) || !isfinite(d->scale)) return GVA_ERR_INVALID_ARG;
  if (d->d_r > 0 && (!(d->rope_base > 0.0) || !isfinite(d->rope_base))) return GVA_ERR_INVALID_ARG;
  if (d->d_c + d->d_r < 1) return GVA_ERR_INVALID_ARG;
  return GVA_OK;
}

inline size_t elem_size(const gva_dims* d) { return d->dtype == GVA_DTYPE_BF16 ? 2 : 4; }

// The tiled cache layout needs whole layout tiles and whole 16-byte pieces.
inline int check_cache_layout(const gva_dims* d) {
  const int piece = (int)(16 / elem_size(d));
  if (d->t_max % kLayoutRows != 0) return GVA_ERR_UNSUPPORTED;
  if (d->d_v % piece != 0 || d->d_r % piece != 0) return GVA_ERR_UNSUPPORTED;
  if (d->d_r / 2 > kMaxPairs) return GVA_ERR_UNSUPPORTED;
  // buffer offsets are 32-bit; keep headroom for prefetches past the end
  const double stream_bytes = (double)d->t_max * (double)(d->d_v > d->d_r ? d->d_v : d->d_r) * elem_size(d);
  if (stream_bytes >= 2147483648.0 - 16777216.0) return GVA_ERR_UNSUPPORTED;
  return GVA_OK;
}

inline void fill_inv_freq(const gva_dims* d, double* out) {
  for (int i = 0; i < kMaxPairs; ++i)
    out[i] = (i < d->d_r / 2) ? pow(d->rope_base, -2.0 * (double)i / (double)d->d_r) : 0.0;
}

inline float scale_log2(const gva_dims* d) {
  const double sc = d->scale > 0.0 ? d->scale : 1.0 / sqrt((double)(d->d_c + d->d_r));
  return (float)(sc * kLog2e);
}

// Workgroups of a decode launch (see work_item).
inline long long decode_grid(const gva_dims* d, int num_splits, int split_rows) {
  const long long slots = (long long)d->batch * num_splits;
  return d->n_groups * (split_rows > 0 ? (slots + 7LL) & ~7LL : slots);
}

// Compute units of the current device (256 if the runtime cannot say).
inline int device_cu_count() {
  int dev = 0, cu = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cu > 0)
    return cu;
  return 256;
}

inline int launch_status() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? GVA_OK : GVA_ERR_HIP;
}

}  // namespace
