// libgva.so -- causal prefill of GVA (Algorithm 1 for every prompt position at
// once): prefill_bf16_kernel (the waves of a workgroup split its key tiles),
// prefill_vt_kernel (the waves split its columns and share each tile's V^T),
// gva_prefill_attention and the matched-GQA baseline gva_gqa_prefill_attention.

#include "gva_common.h"

namespace {

// =============================================================== prefill
// Causal attention for the last N cached rows of every sequence (a prompt,
// after any cached prefix): query i of sequence b sits at position
// p = L_b - N + i and sees rows 0..p (Algorithm 1's loop for every prompt
// position at once; Section 3.3's absorbed scores).  Unlike a decode step
// this is a dense contraction: a workgroup takes C (position, head)
// columns of one group -- C / (H/G) consecutive positions times the H/G
// heads that share the group's value rows; C = 64, or 32 at d_v = 128 to
// stay within 256 registers -- and its four waves split the key tiles up to
// the block's last position.  Per 32-row key tile a wave forms the scores
// of all C columns on the matrix cores (keys = [V | k_r] rows as stored),
// masks rows past each column's position, updates the online softmax and
// accumulates P.V (V transposed once per tile with the identity MFMA,
// shared by the column blocks).
// Precision.  The absorbed and rotated queries enter the score product as
// bf16 high + low pairs (x = hi + lo to ~2^-16 of x, as in the decode
// kernel): a single bf16 query moves every logit by up to 2^-9 of its size,
// an error that grows with the sharpness of the scores.  The high parts
// stay in registers; the low parts, the same for every tile and every wave
// of the workgroup, are read from LDS each tile (registers are the limit).
// A positional slice of at most 16 entries fills half of its 32-wide
// K-chunk, so its low part rides in the other half of the same product.
// P.V runs in fp16: the transposed rows come out of the identity product in
// fp32 and every bf16 value of magnitude 2^-14 .. 65504 is exact in fp16,
// while the weights in [0, 1] keep 3 more bits than bf16.
// The waves merge through LDS.
// Query blocks are dealt longest first, so the triangle's tail is short.
// GQA = true is the matched grouped-query prefill the paper compares
// against: scores read an explicit key stream, no positional term; its
// queries take the same high + low pairs.
// (position, head) columns per workgroup: 64, fewer where a wider value
// row (or the baseline's separate key tile) needs the registers
__host__ __device__ constexpr int prefill_cols(int dv, bool gqa) { return dv >= 128 ? (gqa ? 16 : 32) : 64; }

struct PrefillParams {
  const float* q_abs;     // [B][N][H][d_v]: absorbed queries (GQA: the raw query)
  const float* q_rot;     // [B][N][H][d_r]: rotated positional queries
  const void* v;          // tiled caches, the prompt's rows already appended
  const void* kr;
  const void* k_gqa;      // matched-GQA baseline: explicit key stream (tiled like v)
  const int32_t* lens;
  float* o;               // [B][N][H][d_v]
  float* lse;             // [B][N][H]
  int32_t B, H, G, N, d_r, t_max, n_qblocks;
  float scale_log2;
};

constexpr float kLazyMax = 8.f;

// Two workgroups per CU where the registers allow it without spilling.
constexpr int prefill_min_blocks(int nrc) { return nrc >= 2 ? 1 : 2; }

// KPACK: the positional slice has at most 16 entries (one K-chunk, half
// used), so its low part shares that chunk.
template <int HPG, int DV, int NRC, bool GQA, bool KPACK>
__global__ void __launch_bounds__(kThreads, prefill_min_blocks(NRC)) prefill_bf16_kernel(PrefillParams p) {
  static_assert(!KPACK || NRC == 1, "a packed positional chunk is a single chunk");
  constexpr int COLS = prefill_cols(DV, GQA), NC = DV / 32, NB = DV / 16, CB = COLS / 16;
  constexpr int QB = COLS / HPG;               // positions per workgroup
  constexpr int DEPTH = 2;
  constexpr int RS = DV + 2;                   // per-(wave, column) record: [m, l, o[DV]]
  constexpr int NLO = NC + (KPACK ? 0 : NRC);  // low-part K-chunks read from LDS per column block
  constexpr int RED_FLOATS = kWaves * COLS * RS;
  constexpr int LO_FLOATS = CB * NLO * 64 * 4; // bf16x8 per lane, [cb][chunk][lane]
  // the low parts are read during the key loop, the records only after it
  __shared__ __attribute__((aligned(16))) float lds[RED_FLOATS > LO_FLOATS ? RED_FLOATS : LO_FLOATS];
  float* red = lds;
  bf16x8* lo_lds = reinterpret_cast<bf16x8*>(lds);

  const int nbg = p.B * p.G;
  const int x = blockIdx.x;
  const int qb = p.n_qblocks - 1 - x / nbg;    // longest query blocks first
  const int b = (x % nbg) / p.G, g = (x % nbg) % p.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, qd = lane >> 4;
  const int h0 = g * HPG;
  const bf16x8 zero8 = as_bf16x8(u32x4{0u, 0u, 0u, 0u});

  const int L = clamp_len(p.lens, b, p.t_max);
  const int i_end = min(p.N, (qb + 1) * QB);
  const int kend = L - p.N + i_end;            // rows the block's last position sees
  // column 16 cb + n of this lane: position i = qb QB + col / HPG, head
  // h0 + col % HPG; pos[cb] = its position, or -1 if it has none
  int pos[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int col = 16 * cb + n;
    const int i = qb * QB + col / HPG;
    const int ps = L - p.N + i;
    pos[cb] = (i < p.N && ps >= 0) ? ps : -1;
  }
  const int p_first = L - p.N + qb * QB;       // the block's first position

  // ---- key tiles: rows [0, kend), read through descriptors that end at
  // the last layout tile (reads past it return zeros)
  const int kend16 = kend > 0 ? ((kend + kLayoutRows - 1) / kLayoutRows) * kLayoutRows : 0;
  const uint16_t* vbase = static_cast<const uint16_t*>(p.v) + ((int64_t)b * p.G + g) * p.t_max * DV;
  const uint16_t* kbase = static_cast<const uint16_t*>(p.kr) + (int64_t)b * p.t_max * p.d_r;
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(vbase), (short)0, kend16 * DV * 2, kBufferWord3);
  const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(kbase), (short)0, NRC > 0 ? kend16 * p.d_r * 2 : 0, kBufferWord3);
  const __amdgpu_buffer_rsrc_t kcres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(GQA ? static_cast<const void*>(static_cast<const uint16_t*>(p.k_gqa) +
                                                       ((int64_t)b * p.G + g) * p.t_max * DV)
                            : static_cast<const void*>(vbase)),
      (short)0, kend16 * DV * 2, kBufferWord3);
  const int kpieces = p.d_r / 8;
  const int v_lane = qd * 256 + n * 16;
  // positional K-slots: piece qd of the row (lanes past d_r re-read a valid
  // piece against a zero query); packed, slots kpieces .. 2 kpieces - 1
  // repeat the row's pieces for the query's low part
  int k_lane[NRC > 0 ? NRC : 1];
#pragma unroll
  for (int rc = 0; rc < NRC; ++rc) {
    const int piece = KPACK ? (qd < 2 * kpieces ? qd % kpieces : 0) : min(4 * rc + qd, kpieces - 1);
    k_lane[rc] = piece * 256 + n * 16;
  }
  const int v_tile_bytes = 16 * DV * 2, k_tile_bytes = 16 * p.d_r * 2;
  const int ntiles = kend > 0 ? (kend + kTileRows - 1) / kTileRows : 0;
  const int my_tiles = ntiles > w ? (ntiles - w + kWaves - 1) / kWaves : 0;
  auto tile_row = [&](int j) { return (w + kWaves * j) * kTileRows; };
  using TileT = Tile<DV, NRC, GQA>;
  auto load_tile = [&](TileT& t, int row0) {
    const int lt = row0 / kLayoutRows;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int vsoff = (lt + hf) * v_tile_bytes;
      if constexpr (GQA) {
#pragma unroll
        for (int c = 0; c < NC; ++c)
          t.kc[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(kcres, v_lane + 1024 * c, vsoff, 0));
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
        t.v[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(vres, v_lane + 1024 * c, vsoff, 0));
#pragma unroll
      for (int rc = 0; rc < NRC; ++rc)
        t.k[hf][rc] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(kres, k_lane[rc], (lt + hf) * k_tile_bytes, 0));
    }
  };
  TileT buf[DEPTH];
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d) {
    load_tile(buf[d], tile_row(d));
    __builtin_amdgcn_sched_barrier(0);
  }

  // ---- the queries as bf16 high + low B operands (zero for columns with
  // no position).  Every wave forms the high parts of all the workgroup's
  // columns; the low parts go to LDS, each chunk written by one wave.
  bf16x8 bq[CB][NC];
  bf16x8 bk[CB][NRC > 0 ? NRC : 1];
  auto put_lo = [&](int cb, int c, const float* xv, bool live) {
    if ((cb * NLO + c) % kWaves == w) lo_lds[(cb * NLO + c) * 64 + lane] = live ? split_hi_lo(xv, true) : zero8;
  };
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int col = 16 * cb + n;
    const int i = min(qb * QB + col / HPG, p.N - 1);
    const int64_t qrow = ((int64_t)b * p.N + i) * p.H + h0 + col % HPG;
    const float* qa = p.q_abs + qrow * DV + 8 * qd;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const f32x4 u0 = *reinterpret_cast<const f32x4*>(qa + 32 * c);
      const f32x4 u1 = *reinterpret_cast<const f32x4*>(qa + 32 * c + 4);
      float xv[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xv[j] = u0[j] * p.scale_log2;
        xv[4 + j] = u1[j] * p.scale_log2;
      }
      bq[cb][c] = pos[cb] >= 0 ? split_hi_lo(xv, false) : zero8;
      put_lo(cb, c, xv, pos[cb] >= 0);
    }
#pragma unroll
    for (int rc = 0; rc < NRC; ++rc) {
      // the positional piece this lane's K-slot carries: high part of piece
      // 4 rc + qd, or (packed) the low part of piece qd - kpieces
      const bool hi_slot = KPACK ? qd < kpieces : 32 * rc + 8 * qd < p.d_r;
      const bool lo_slot = KPACK && qd >= kpieces && qd < 2 * kpieces;
      const int j0 = KPACK ? 8 * (lo_slot ? qd - kpieces : qd) : 32 * rc + 8 * qd;
      float xv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (hi_slot || lo_slot) {
        const float* qr = p.q_rot + qrow * p.d_r + j0;
        const f32x4 u0 = *reinterpret_cast<const f32x4*>(qr);
        const f32x4 u1 = *reinterpret_cast<const f32x4*>(qr + 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          xv[j] = u0[j] * p.scale_log2;
          xv[4 + j] = u1[j] * p.scale_log2;
        }
      }
      bk[cb][rc] = (pos[cb] >= 0 && (hi_slot || lo_slot)) ? split_hi_lo(xv, lo_slot) : zero8;
      if constexpr (!KPACK) put_lo(cb, NC + rc, xv, pos[cb] >= 0 && hi_slot);
    }
  }
  __syncthreads();                             // the low parts are in LDS

  bf16x8 esel[2];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    u32x4 u = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (8 * qd + j == n + 16 * half) u[j >> 1] |= 0x3F80u << (16 * (j & 1));
    esel[half] = as_bf16x8(u);
  }

  float m_run[CB], l_run[CB];
  f32x4 acc[CB][NB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    m_run[cb] = -INFINITY;
    l_run[cb] = 0.f;
#pragma unroll
    for (int ib = 0; ib < NB; ++ib) acc[cb][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto compute_tile = [&](TileT& t, int row0) {
    if (row0 + kTileRows > kend) {             // rows past the block's keys: zero
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bool dead = row0 + 16 * hf + n >= kend;
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
    const bool masked = row0 + kTileRows - 1 > p_first;   // some column may not see every row
    // the LDS offset is opaque to the compiler, so the low parts are read
    // here, tile by tile, instead of being hoisted into registers
    int lo_off = lane;
    asm volatile("" : "+v"(lo_off));
    // scores of one column block: the high and the low query parts
    // accumulate into one sum per 16-row half
    auto scores = [&](int cb, f32x4 (&sc)[2]) {
      bf16x8 lo[NLO];
#pragma unroll
      for (int c = 0; c < NLO; ++c) lo[c] = lo_lds[(cb * NLO + c) * 64 + lo_off];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        sc[hf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          sc[hf] = mfma16(GQA ? t.kc[hf][c] : t.v[hf][c], bq[cb][c], sc[hf]);
          sc[hf] = mfma16(GQA ? t.kc[hf][c] : t.v[hf][c], lo[c], sc[hf]);
        }
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc) {
          sc[hf] = mfma16(t.k[hf][rc], bk[cb][rc], sc[hf]);
          if constexpr (!KPACK) sc[hf] = mfma16(t.k[hf][rc], lo[NC + rc], sc[hf]);
        }
      }
    };
    // the online softmax of one column block, its weights as fp16
    auto softmax = [&](int cb, const f32x4 (&sc)[2]) {
      float xv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) xv[k] = sc[k >> 2][k & 3];
      if (masked) {
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (row0 + 16 * (k >> 2) + 4 * qd + (k & 3) > pos[cb]) xv[k] = -INFINITY;
      }
      float mt = xv[0];
#pragma unroll
      for (int k = 1; k < 8; ++k) mt = fmaxf(mt, xv[k]);
      mt = max_over_rows(mt);
      const float m_new = fmaxf(m_run[cb], mt);
      // The running maximum moves only once some column's tile maximum
      // exceeds it by more than kLazyMax (log2 units): the weights then stay
      // below 2^kLazyMax (fp16 holds them; the sums are fp32), and the
      // accumulators are rescaled on few tiles.
      if (__ballot(mt > m_run[cb] + kLazyMax) != 0) {
        // columns whose rows so far are all masked keep m = -inf: scale 1
        const float alpha = m_new > m_run[cb] ? __builtin_amdgcn_exp2f(m_run[cb] - m_new) : 1.f;
        l_run[cb] *= alpha;
#pragma unroll
        for (int ib = 0; ib < NB; ++ib) acc[cb][ib] *= alpha;
        m_run[cb] = m_new;
      }
      const float m_use = m_run[cb] == -INFINITY ? 0.f : m_run[cb];   // all masked so far
      float pr[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        pr[k] = __builtin_amdgcn_exp2f(xv[k] - m_use);
        l_run[cb] += pr[k];
      }
      return to_f16x8(pr);
    };
    // The next column block's score products are issued before this
    // block's softmax, so the matrix cores run them while the vector units
    // work (the order is pinned by scheduling barriers).
    f16x8 bp[CB];
    f32x4 sc[2][2];
    scores(0, sc[0]);
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      if (cb + 1 < CB) scores(cb + 1, sc[(cb + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
      bp[cb] = softmax(cb, sc[cb & 1]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // P.V over the 2 NC 16-wide output blocks; the identity products that
    // transpose block k + 1 of V are issued before block k's conversion to
    // fp16 and its products
    auto transpose = [&](int k, f32x4 (&tq)[2]) {
      const int c = k >> 1, half = k & 1;
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      tq[0] = mfma16(t.v[0][c], esel[half], z);
      tq[1] = mfma16(t.v[1][c], esel[half], z);
    };
    f32x4 tq[2][2];
    transpose(0, tq[0]);
#pragma unroll
    for (int k = 0; k < 2 * NC; ++k) {
      if (k + 1 < 2 * NC) transpose(k + 1, tq[(k + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
      const f32x4* tk = tq[k & 1];
      const float tv[8] = {tk[0][0], tk[0][1], tk[0][2], tk[0][3], tk[1][0], tk[1][1], tk[1][2], tk[1][3]};
      const f16x8 av = to_f16x8(tv);           // bf16 values: exact in fp16 at these magnitudes
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[cb][k] = mfma16(av, bp[cb], acc[cb][k]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  for (int jt = 0; jt < my_tiles; jt += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int j = jt + d;
      if (j >= my_tiles) break;
      load_tile(buf[(d + DEPTH - 1) % DEPTH], tile_row(j + DEPTH - 1));
      __builtin_amdgcn_sched_barrier(0);
      compute_tile(buf[d], tile_row(j));
    }
  }

  // ---- merge the waves: per column the records (m, l, o) of the 4 waves
  __syncthreads();                             // every wave is done with the low parts
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const float l = sum_over_rows(l_run[cb]);
    float* rec = red + (w * COLS + 16 * cb + n) * RS;
    if (qd == 0) {
      rec[0] = m_run[cb];
      rec[1] = l;
    }
#pragma unroll
    for (int ib = 0; ib < NB; ++ib)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) rec[2 + 16 * ib + 4 * qd + jj] = acc[cb][ib][jj];
  }
  __syncthreads();
  for (int idx = tid; idx < COLS * DV; idx += kThreads) {
    const int col = idx / DV, i = idx % DV;
    const int qi = qb * QB + col / HPG;
    if (qi >= p.N) continue;
    float mx = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) mx = fmaxf(mx, red[(ww * COLS + col) * RS]);
    float o = 0.f, lsum = 0.f;
    if (mx != -INFINITY && L - p.N + qi >= 0) {
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww) {
        const float* rec = red + (ww * COLS + col) * RS;
        if (rec[0] == -INFINITY) continue;       // this wave saw no row of the column
        const float sc = __builtin_amdgcn_exp2f(rec[0] - mx);
        lsum += rec[1] * sc;
        o += rec[2 + i] * sc;
      }
      o /= lsum;
    } else {
      mx = -INFINITY;
    }
    const int64_t orow = ((int64_t)b * p.N + qi) * p.H + h0 + col % HPG;
    __builtin_nontemporal_store(o, p.o + orow * DV + i);   // written once: kept out of the L2
    if (i == 0) p.lse[orow] = mx == -INFINITY ? -INFINITY : (mx + log2f(lsum)) * kLn2;
  }
}

// ----------------------------------------------- prefill, columns per wave
// The same causal prefill with the work divided the other way: each of the
// four waves owns CW (position, head) columns of its own and walks every
// key tile of the workgroup's range, so the waves hold disjoint softmax
// states and write their own outputs (no merge).  All four waves work on
// one key tile at a time and share its V^T: wave w transposes NB / 4 of
// the tile's 16-wide value blocks (identity products, fp16) into LDS, and
// after one barrier every wave reads all NB blocks for its P.V.  Per tile a
// wave then issues a quarter of the identity products (2 NB / 4 instead of
// 2 NB) and converts a quarter of the blocks to fp16; the V tile itself is
// read by all four waves from the cache hierarchy (the same rows at the
// same time).
// Columns per wave: 32, or 16 for the matched-GQA baseline, whose separate
// key tile takes the registers of the second column block.
__host__ __device__ constexpr int prefill_vt_cols(int dv, bool gqa) { return gqa ? 16 : (dv >= 128 ? 32 : 64); }

template <int HPG, int DV, int NRC, bool GQA, bool KPACK>
__global__ void __launch_bounds__(kThreads, 2) prefill_vt_kernel(PrefillParams p) {
  static_assert(!KPACK || NRC == 1, "a packed positional chunk is a single chunk");
  static_assert(!GQA || NRC == 0, "the GQA baseline has no positional term");
  constexpr int CW = prefill_vt_cols(DV, GQA), NC = DV / 32, NB = DV / 16, CB = CW / 16;
  constexpr int WCOLS = kWaves * CW;           // columns per workgroup
  constexpr int QB = WCOLS / HPG;              // positions per workgroup
  constexpr int KPW = NB / kWaves;             // V^T blocks each wave transposes
  static_assert(KPW >= 1 && NB % kWaves == 0, "every wave transposes whole blocks");
  constexpr int DEPTH = 2;
  constexpr int NLO = NC + (KPACK ? 0 : NRC);
  // P.V one tile behind the scores (below), except in the matched-GQA
  // baseline, which ran slower so; kAhead column blocks' scores are issued
  // before that P.V: one where a separate positional chunk and its low parts
  // already hold the registers (all of them would spill), else all
  constexpr bool kPipe = !GQA;
  constexpr int kAhead = (NRC > 0 && !KPACK) ? 1 : CB;
  __shared__ bf16x8 lo_lds[kWaves * CB * NLO * 64];   // the low query parts, per wave
  __shared__ f16x8 vt_lds[2 * NB * 64];               // V^T blocks of a tile, two buffers

  const int nbg = p.B * p.G;
  const int x = blockIdx.x;
  const int qb = p.n_qblocks - 1 - x / nbg;    // longest query blocks first
  const int b = (x % nbg) / p.G, g = (x % nbg) % p.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, qd = lane >> 4;
  const int h0 = g * HPG;
  const bf16x8 zero8 = as_bf16x8(u32x4{0u, 0u, 0u, 0u});

  const int L = clamp_len(p.lens, b, p.t_max);
  const int i_end = min(p.N, (qb + 1) * QB);
  const int kend = L - p.N + i_end;            // rows the block's last position sees
  // column CW w + 16 cb + n of this lane: position i = qb QB + col / HPG,
  // head h0 + col % HPG; pos[cb] = its position, or -1 if it has none
  int pos[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int col = CW * w + 16 * cb + n;
    const int i = qb * QB + col / HPG;
    const int ps = L - p.N + i;
    pos[cb] = (i < p.N && ps >= 0) ? ps : -1;
  }
  const int p_first = L - p.N + qb * QB + (CW * w) / HPG;   // this wave's first position

  // ---- key tiles: rows [0, kend), every wave all of them
  const int kend16 = kend > 0 ? ((kend + kLayoutRows - 1) / kLayoutRows) * kLayoutRows : 0;
  const uint16_t* vbase = static_cast<const uint16_t*>(p.v) + ((int64_t)b * p.G + g) * p.t_max * DV;
  const uint16_t* kbase = static_cast<const uint16_t*>(p.kr) + (int64_t)b * p.t_max * p.d_r;
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(vbase), (short)0, kend16 * DV * 2, kBufferWord3);
  const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(kbase), (short)0, NRC > 0 ? kend16 * p.d_r * 2 : 0, kBufferWord3);
  const __amdgpu_buffer_rsrc_t kcres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(GQA ? static_cast<const void*>(static_cast<const uint16_t*>(p.k_gqa) +
                                                       ((int64_t)b * p.G + g) * p.t_max * DV)
                            : static_cast<const void*>(vbase)),
      (short)0, kend16 * DV * 2, kBufferWord3);
  const int kpieces = p.d_r / 8;
  const int v_lane = qd * 256 + n * 16;
  int k_lane[NRC > 0 ? NRC : 1];
#pragma unroll
  for (int rc = 0; rc < NRC; ++rc) {
    const int piece = KPACK ? (qd < 2 * kpieces ? qd % kpieces : 0) : min(4 * rc + qd, kpieces - 1);
    k_lane[rc] = piece * 256 + n * 16;
  }
  const int v_tile_bytes = 16 * DV * 2, k_tile_bytes = 16 * p.d_r * 2;
  const int ntiles = kend > 0 ? (kend + kTileRows - 1) / kTileRows : 0;
  using TileT = Tile<DV, NRC, GQA>;
  auto load_tile = [&](TileT& t, int row0) {
    const int lt = row0 / kLayoutRows;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int vsoff = (lt + hf) * v_tile_bytes;
      if constexpr (GQA) {
#pragma unroll
        for (int c = 0; c < NC; ++c)
          t.kc[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(kcres, v_lane + 1024 * c, vsoff, 0));
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
        t.v[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(vres, v_lane + 1024 * c, vsoff, 0));
#pragma unroll
      for (int rc = 0; rc < NRC; ++rc)
        t.k[hf][rc] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(kres, k_lane[rc], (lt + hf) * k_tile_bytes, 0));
    }
  };
  TileT buf[DEPTH];
  load_tile(buf[0], 0);
  load_tile(buf[1], kTileRows);
  __builtin_amdgcn_sched_barrier(0);

  // ---- this wave's queries as bf16 high + low B operands (zero for columns
  // with no position); the low parts to this wave's LDS region
  bf16x8 bq[CB][NC];
  bf16x8 bk[CB][NRC > 0 ? NRC : 1];
  bf16x8* my_lo = lo_lds + w * (CB * NLO * 64);
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int col = CW * w + 16 * cb + n;
    const int i = min(qb * QB + col / HPG, p.N - 1);
    const int64_t qrow = ((int64_t)b * p.N + i) * p.H + h0 + col % HPG;
    const float* qa = p.q_abs + qrow * DV + 8 * qd;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const f32x4 u0 = *reinterpret_cast<const f32x4*>(qa + 32 * c);
      const f32x4 u1 = *reinterpret_cast<const f32x4*>(qa + 32 * c + 4);
      float xv[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xv[j] = u0[j] * p.scale_log2;
        xv[4 + j] = u1[j] * p.scale_log2;
      }
      bq[cb][c] = pos[cb] >= 0 ? split_hi_lo(xv, false) : zero8;
      my_lo[(cb * NLO + c) * 64 + lane] = pos[cb] >= 0 ? split_hi_lo(xv, true) : zero8;
    }
#pragma unroll
    for (int rc = 0; rc < NRC; ++rc) {
      const bool hi_slot = KPACK ? qd < kpieces : 32 * rc + 8 * qd < p.d_r;
      const bool lo_slot = KPACK && qd >= kpieces && qd < 2 * kpieces;
      const int j0 = KPACK ? 8 * (lo_slot ? qd - kpieces : qd) : 32 * rc + 8 * qd;
      float xv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (hi_slot || lo_slot) {
        const float* qr = p.q_rot + qrow * p.d_r + j0;
        const f32x4 u0 = *reinterpret_cast<const f32x4*>(qr);
        const f32x4 u1 = *reinterpret_cast<const f32x4*>(qr + 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          xv[j] = u0[j] * p.scale_log2;
          xv[4 + j] = u1[j] * p.scale_log2;
        }
      }
      bk[cb][rc] = (pos[cb] >= 0 && (hi_slot || lo_slot)) ? split_hi_lo(xv, lo_slot) : zero8;
      if constexpr (!KPACK)
        my_lo[(cb * NLO + NC + rc) * 64 + lane] = (pos[cb] >= 0 && hi_slot) ? split_hi_lo(xv, true) : zero8;
    }
  }

  bf16x8 esel[2];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    u32x4 u = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (8 * qd + j == n + 16 * half) u[j >> 1] |= 0x3F80u << (16 * (j & 1));
    esel[half] = as_bf16x8(u);
  }

  float m_run[CB], l_run[CB];
  f32x4 acc[CB][NB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    m_run[cb] = -INFINITY;
    l_run[cb] = 0.f;
#pragma unroll
    for (int ib = 0; ib < NB; ++ib) acc[cb][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  f16x8 bp_prev[CB];                           // the previous tile's weights (pipelined P.V)
  // next_row: the tile requested into t's registers once its scores are issued
  auto compute_tile = [&](TileT& t, int row0, int vbuf, bool has_prev, int next_row) {
    if (row0 + kTileRows > kend) {             // rows past the block's keys: zero
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bool dead = row0 + 16 * hf + n >= kend;
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
    // this wave's share of the tile's V^T, into LDS first: the other waves
    // read it after the barrier below
    f16x8* vt = vt_lds + vbuf * (NB * 64);
#pragma unroll
    for (int kk = 0; kk < KPW; ++kk) {
      const int k = w * KPW + kk;              // 16-wide value block k: chunk k / 2, half k % 2
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      f32x4 t0 = z, t1 = z;
      const bf16x8 e = (k & 1) ? esel[1] : esel[0];
#pragma unroll
      for (int c = 0; c < NC; ++c)
        if (c == (k >> 1)) {
          t0 = mfma16(t.v[0][c], e, z);
          t1 = mfma16(t.v[1][c], e, z);
        }
      const float tv[8] = {t0[0], t0[1], t0[2], t0[3], t1[0], t1[1], t1[2], t1[3]};
      vt[k * 64 + lane] = to_f16x8(tv);       // bf16 values: exact in fp16 at these magnitudes
    }
    const bool masked = row0 + kTileRows - 1 > p_first;   // some column may not see every row
    int lo_off = lane;
    asm volatile("" : "+v"(lo_off));
    auto scores = [&](int cb, f32x4 (&sc)[2]) {
      bf16x8 lo[NLO];
#pragma unroll
      for (int c = 0; c < NLO; ++c) lo[c] = my_lo[(cb * NLO + c) * 64 + lo_off];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        sc[hf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          sc[hf] = mfma16(GQA ? t.kc[hf][c] : t.v[hf][c], bq[cb][c], sc[hf]);
          sc[hf] = mfma16(GQA ? t.kc[hf][c] : t.v[hf][c], lo[c], sc[hf]);
        }
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc) {
          sc[hf] = mfma16(t.k[hf][rc], bk[cb][rc], sc[hf]);
          if constexpr (!KPACK) sc[hf] = mfma16(t.k[hf][rc], lo[NC + rc], sc[hf]);
        }
      }
    };
    auto softmax = [&](int cb, const f32x4 (&sc)[2]) {
      float xv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) xv[k] = sc[k >> 2][k & 3];
      if (masked) {
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (row0 + 16 * (k >> 2) + 4 * qd + (k & 3) > pos[cb]) xv[k] = -INFINITY;
      }
      float mt = xv[0];
#pragma unroll
      for (int k = 1; k < 8; ++k) mt = fmaxf(mt, xv[k]);
      mt = max_over_rows(mt);
      const float m_new = fmaxf(m_run[cb], mt);
      if (__ballot(mt > m_run[cb] + kLazyMax) != 0) {
        const float alpha = m_new > m_run[cb] ? __builtin_amdgcn_exp2f(m_run[cb] - m_new) : 1.f;
        l_run[cb] *= alpha;
#pragma unroll
        for (int ib = 0; ib < NB; ++ib) acc[cb][ib] *= alpha;
        m_run[cb] = m_new;
      }
      const float m_use = m_run[cb] == -INFINITY ? 0.f : m_run[cb];
      float pr[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        pr[k] = __builtin_amdgcn_exp2f(xv[k] - m_use);
        l_run[cb] += pr[k];
      }
      return to_f16x8(pr);
    };
    if constexpr (kPipe) {
      // P.V of the previous tile (its V^T in the other buffer, complete since
      // the previous barrier) is issued with this tile's softmax, so the
      // matrix cores run it while the vector units work; it comes first in
      // program order, before any rescale of the accumulators
      f32x4 sc[CB][2];
#pragma unroll
      for (int cb = 0; cb < kAhead; ++cb) scores(cb, sc[cb]);
      if constexpr (kAhead == CB) load_tile(t, next_row);
      __builtin_amdgcn_sched_barrier(0);
      if (has_prev) {
        const f16x8* vtp = vt_lds + (vbuf ^ 1) * (NB * 64);
#pragma unroll
        for (int k = 0; k < NB; ++k) {
          const f16x8 av = vtp[k * 64 + lane];
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) acc[cb][k] = mfma16(av, bp_prev[cb], acc[cb][k]);
        }
      }
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        if (cb >= kAhead) {
          __builtin_amdgcn_sched_barrier(0);
          scores(cb, sc[cb]);
          __builtin_amdgcn_sched_barrier(0);
        }
        bp_prev[cb] = softmax(cb, sc[cb]);
      }
      if constexpr (kAhead < CB) load_tile(t, next_row);
      __syncthreads();                         // every wave's V^T blocks of this tile are in LDS
    } else {
      f16x8 bp[CB];
      f32x4 sc[2][2];
      scores(0, sc[0]);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        if (cb + 1 < CB) scores(cb + 1, sc[(cb + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        bp[cb] = softmax(cb, sc[cb & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
      load_tile(t, next_row);
      __syncthreads();                         // every wave's V^T blocks of this tile are in LDS
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const f16x8 av = vt[k * 64 + lane];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) acc[cb][k] = mfma16(av, bp[cb], acc[cb][k]);
      }
    }
  };

  // Every wave runs every tile (the barrier inside compute_tile is reached
  // the same number of times by all four); tile j + 2 is requested into
  // tile j's registers as soon as tile j's scores no longer need them.
  // (requests past the block's rows read zeros through the descriptors and
  // cost no traffic, so they are unconditional and the waits exact)
  for (int jt = 0; jt < ntiles; jt += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int j = jt + d;
      if (j >= ntiles) break;
      compute_tile(buf[d], j * kTileRows, d, j > 0, (j + DEPTH) * kTileRows);
    }
  }
  if (kPipe && ntiles > 0) {                   // P.V of the last tile
    const f16x8* vtl = vt_lds + ((ntiles - 1) & 1) * (NB * 64);
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const f16x8 av = vtl[k * 64 + lane];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[cb][k] = mfma16(av, bp_prev[cb], acc[cb][k]);
    }
  }

  // ---- this wave's columns: normalise and write
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const float l = sum_over_rows(l_run[cb]);
    const int col = CW * w + 16 * cb + n;
    const int qi = qb * QB + col / HPG;
    if (qi >= p.N) continue;
    const bool seen = m_run[cb] != -INFINITY && L - p.N + qi >= 0;
    const float inv = seen ? 1.f / l : 0.f;
    const int64_t orow = ((int64_t)b * p.N + qi) * p.H + h0 + col % HPG;
#pragma unroll
    for (int ib = 0; ib < NB; ++ib) {
      f32x4 o = acc[cb][ib] * inv;
      // written once and not read again here: kept out of the L2, which holds
      // the group's key and value rows
      __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(p.o + orow * DV + 16 * ib + 4 * qd));
    }
    if (qd == 0) p.lse[orow] = seen ? (m_run[cb] + log2f(l)) * kLn2 : -INFINITY;
  }
}

using PrefillFn = void (*)(PrefillParams);

template <int HPG, int DV>
PrefillFn pick_prefill_nrc(int d_r, bool gqa) {
  if (gqa) return prefill_bf16_kernel<HPG, DV, 0, true, false>;
  if (d_r == 0) return prefill_bf16_kernel<HPG, DV, 0, false, false>;
  if (d_r <= 16) return prefill_bf16_kernel<HPG, DV, 1, false, true>;
  if (d_r <= 32) return prefill_bf16_kernel<HPG, DV, 1, false, false>;
  if (d_r <= 64) return prefill_bf16_kernel<HPG, DV, 2, false, false>;
  return nullptr;
}

template <int HPG>
PrefillFn pick_prefill_dv(int dv, int d_r, bool gqa) {
  switch (dv) {
    case 64: return pick_prefill_nrc<HPG, 64>(d_r, gqa);
    case 128: return pick_prefill_nrc<HPG, 128>(d_r, gqa);
  }
  return nullptr;
}

PrefillFn pick_prefill(int hpg, int dv, int d_r, bool gqa) {
  switch (hpg) {
    case 1: return pick_prefill_dv<1>(dv, d_r, gqa);
    case 2: return pick_prefill_dv<2>(dv, d_r, gqa);
    case 4: return pick_prefill_dv<4>(dv, d_r, gqa);
    case 8: return pick_prefill_dv<8>(dv, d_r, gqa);
  }
  return nullptr;
}

template <int HPG, int DV>
PrefillFn pick_prefill_vt_nrc(int d_r) {
  if (d_r == 0) return prefill_vt_kernel<HPG, DV, 0, false, false>;
  if (d_r <= 16) return prefill_vt_kernel<HPG, DV, 1, false, true>;
  if (d_r <= 32) return prefill_vt_kernel<HPG, DV, 1, false, false>;
  return nullptr;                              // two positional chunks: the tile-split kernel
}

PrefillFn pick_prefill_vt(int hpg, int dv, int d_r, bool gqa) {
  if (dv != 128) return nullptr;               // d_v = 64: the tile-split kernel (measured faster)
  switch (hpg) {
    case 1: return gqa ? prefill_vt_kernel<1, 128, 0, true, false> : pick_prefill_vt_nrc<1, 128>(d_r);
    case 2: return gqa ? prefill_vt_kernel<2, 128, 0, true, false> : pick_prefill_vt_nrc<2, 128>(d_r);
    case 4: return gqa ? prefill_vt_kernel<4, 128, 0, true, false> : pick_prefill_vt_nrc<4, 128>(d_r);
    case 8: return gqa ? prefill_vt_kernel<8, 128, 0, true, false> : pick_prefill_vt_nrc<8, 128>(d_r);
  }
  return nullptr;
}

// The columns-per-wave kernel has a quarter of the workgroups of the
// tile-split one; it wins once they fill the GPU a few times over: from
// two per CU (H/G <= 4) or four per CU (H/G = 8), measured on prompts of
// 1K-16K tokens at d_v = 128.
bool prefer_prefill_vt(const gva_dims* d, int n_new, bool gqa) {
  const int hpg = d->n_heads / d->n_groups;
  const int qb = kWaves * prefill_vt_cols(d->d_v, gqa) / hpg;   // positions per workgroup
  if (qb < 1) return false;
  const long long qblocks = (n_new + qb - 1) / qb;
  const long long items = (long long)d->batch * d->n_groups * qblocks;
  return items >= (hpg >= 8 ? 4LL : 2LL) * device_cu_count();
}

// The launch behind gva_prefill_attention and, with k_gqa given,
// gva_gqa_prefill_attention.
int prefill_impl(const gva_dims* dims, int32_t n_new, const float* q_abs, const float* q_rot,
                 const void* v_cache, const void* kr_cache, const void* k_gqa, const int32_t* lens,
                 float* o, float* lse, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  const bool gqa = k_gqa != nullptr;
  const int d_r = gqa ? 0 : dims->d_r;
  if (n_new < 1 || n_new > dims->t_max) return GVA_ERR_INVALID_ARG;
  if (!q_abs || !v_cache || !lens || !o || !lse) return GVA_ERR_INVALID_ARG;
  if (d_r > 0 && (!q_rot || !kr_cache)) return GVA_ERR_INVALID_ARG;
  if (!aligned(q_abs, 16) || !aligned(v_cache, 16) || !aligned(lens, 4) || !aligned(o, 16) ||
      !aligned(lse, 4) || (d_r > 0 && (!aligned(q_rot, 16) || !aligned(kr_cache, 16))) ||
      (gqa && !aligned(k_gqa, 16)))
    return GVA_ERR_INVALID_ARG;
  if (dims->dtype != GVA_DTYPE_BF16) return GVA_ERR_UNSUPPORTED;
  st = check_cache_layout(dims);
  if (st != GVA_OK) return st;
  if (d_r % 8 != 0 || d_r > 64) return GVA_ERR_UNSUPPORTED;
  const int hpg = dims->n_heads / dims->n_groups;
  // columns per wave where it has a kernel (d_v = 128; GVA with d_r <= 32,
  // or the GQA baseline) and the grid is large enough, else the tile-split
  // kernel (d_v = 64, two positional chunks, short prompts)
  PrefillFn fn = prefer_prefill_vt(dims, n_new, gqa) ? pick_prefill_vt(hpg, dims->d_v, d_r, gqa) : nullptr;
  const bool per_wave = fn != nullptr;
  if (!per_wave) fn = pick_prefill(hpg, dims->d_v, d_r, gqa);
  if (fn == nullptr) return GVA_ERR_UNSUPPORTED;
  const int qb_rows = (per_wave ? kWaves * prefill_vt_cols(dims->d_v, gqa) : prefill_cols(dims->d_v, gqa)) / hpg;
  const long long n_qblocks = (n_new + qb_rows - 1) / qb_rows;
  const long long n_items = (long long)dims->batch * dims->n_groups * n_qblocks;
  if (n_items > 0x7FFFFFFFLL) return GVA_ERR_UNSUPPORTED;

  PrefillParams p{};
  memset(&p, 0, sizeof(p));
  p.q_abs = q_abs;
  p.q_rot = q_rot;
  p.v = v_cache;
  p.kr = kr_cache;
  p.k_gqa = k_gqa;
  p.lens = lens;
  p.o = o;
  p.lse = lse;
  p.B = dims->batch;
  p.H = dims->n_heads;
  p.G = dims->n_groups;
  p.N = n_new;
  p.d_r = d_r;
  p.t_max = dims->t_max;
  p.n_qblocks = (int32_t)n_qblocks;
  if (gqa) {
    const double sc = dims->scale > 0.0 ? dims->scale : 1.0 / sqrt((double)dims->d_v);
    p.scale_log2 = (float)(sc * kLog2e);
  } else {
    p.scale_log2 = scale_log2(dims);
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)n_items), dim3(kThreads), 0, static_cast<hipStream_t>(stream), p);
  return launch_status();
}

// The append behind gva_append_kv and, with paging given, gva_paged_append_kv.
}  // namespace

extern "C" {

int gva_prefill_attention(const gva_dims* dims, int32_t n_new, const float* q_abs, const float* q_rot,
                          const void* v_cache, const void* kr_cache, const int32_t* lens, float* o,
                          float* lse, void* stream) {
  return prefill_impl(dims, n_new, q_abs, q_rot, v_cache, kr_cache, nullptr, lens, o, lse, stream);
}

int gva_gqa_prefill_attention(const gva_dims* dims, int32_t n_new, const float* q, const void* k_cache,
                              const void* v_cache, const int32_t* lens, float* o, float* lse,
                              void* stream) {
  if (k_cache == nullptr) return GVA_ERR_INVALID_ARG;
  return prefill_impl(dims, n_new, q, nullptr, v_cache, nullptr, k_cache, lens, o, lse, stream);
}

}  // extern "C"
