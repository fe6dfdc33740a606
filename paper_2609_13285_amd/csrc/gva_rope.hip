// libgva.so -- GVA decode with ordinary RoPE (the contrast path of Section 3.2):
// keys reconstructed and rotated at their own positions, so M_h cannot be
// absorbed.  rope_decode_kernel and gva_rope_decode_attention.

#include "gva_common.h"

namespace {

// ================================================= decode, ordinary RoPE
// The contrast path of Section 3.2: GVA whose keys k_t = v_t M_h are rotated
// over their whole width at their own position, so M_h cannot be absorbed.
// With the column pairs (2i, 2i+1) of q M-space written as complex numbers,
//   RoPE(q, P) . RoPE(v_t M_h, t) = sum_i a_i cos(theta_i d) + b_i sin(theta_i d)
// for d = t - P, where a_i = v_t . W[:, 2i] and b_i = v_t . W[:, 2i+1] with
//   W[r][2i]   = q_2i M_h[r][2i]   + q_2i+1 M_h[r][2i+1]
//   W[r][2i+1] = q_2i+1 M_h[r][2i] - q_2i M_h[r][2i+1].
// Per 32-row tile the kernel forms (V_tile W_h)^T on the matrix cores (d_v *
// d_c multiply-adds per row and head, as explicit key reconstruction costs),
// so each lane holds one row and four consecutive columns; it weights column
// c by cos or sin of theta_i d and sums the columns (in registers, then over
// the four 16-lane rows): the scores.  A per-wave LDS transpose puts them in
// the layout of the GVA kernel, whose softmax, P.V, splits and merge follow.
// W_h is built in the prologue (fp32, pre-scaled, rounded to bf16) and held
// in LDS in MFMA operand order; the angle is reduced in fp64 at every tile's
// first row and the rest of the tile is offset in fp32.
constexpr int kRopeMaxPairs = 64;          // d_c / 2 <= 64
constexpr int kRopeWaves = 8;              // two waves per SIMD
constexpr int kRopeThreads = 64 * kRopeWaves;

struct RopeDecodeParams {
  DecodeArgs a;                            // q [B][H][d_c], m, v, lens, o_part, lse_part, dims
  double freq_rev[kRopeMaxPairs];          // theta_i / (2 pi): revolutions per position
};

template <int HPG, int DV, int DC>
struct RopeCfg {
  // 16-row blocks in a wave's tile: four (64 rows, so every W piece read
  // from LDS feeds four products; the LDS reads of W bound the kernel at
  // two), or two where eight 128-wide heads leave no registers for them
  static constexpr int HF = (HPG >= 8 && DV >= 128) ? 2 : 4;
  static constexpr int TR = 16 * HF;                       // rows per wave tile
  // tiles in flight per wave: the next one is requested while this one is
  // computed, or, where a second 64-row tile does not fit the registers
  // (128-wide values, or eight heads), each half of it once the P.V has
  // read the same half of this one
  static constexpr int DEPTH = (HF == 4 && (DV >= 128 || HPG * DV >= 512)) ? 1 : 2;
  static constexpr int NC = DV / 32;                       // K-chunks per V row
  static constexpr int NB = DV / 16;                       // 16-wide i-blocks of the output
  static constexpr int NBC = DC / 16;                      // 16-wide column blocks of W
  static constexpr int W_FLOATS = HPG * NC * NBC * 64 * 4; // W in 16-byte pieces
  static constexpr int RED_FLOATS = kRopeWaves * HPG * (DV + 2);
  static constexpr int LDS_FLOATS = W_FLOATS > RED_FLOATS ? W_FLOATS : RED_FLOATS;
  static constexpr int XS_FLOATS = kRopeWaves * HPG * TR;          // score transpose
};

template <int HPG, int DV, int DC>
__global__ void __launch_bounds__(kRopeThreads, 1) rope_decode_kernel(RopeDecodeParams p) {
  const DecodeArgs a = p.a;
  using Cfg = RopeCfg<HPG, DV, DC>;
  constexpr int NC = Cfg::NC, NB = Cfg::NB, NBC = Cfg::NBC;
  constexpr int HF = Cfg::HF, TR = Cfg::TR, RH = HF / 2, DEPTH = Cfg::DEPTH;
  __shared__ __attribute__((aligned(16))) float lds[Cfg::LDS_FLOATS];
  __shared__ __attribute__((aligned(16))) float xs_all[Cfg::XS_FLOATS];
  // RoPE angles in turns as 32-bit fractions (wrap-around is the reduction
  // mod one turn): per wave, pair i's angle theta_i (row0 - P) / (2 pi) at
  // the wave's first tile, and the step from one of its tiles to the next
  __shared__ uint32_t ang_all[kRopeWaves * (DC / 2)];
  __shared__ uint32_t ang_step[DC / 2];
  __shared__ float freq_f[DC / 2];             // theta_i / (2 pi), fp32: offsets within a tile

  int b, s, g;
  bool empty_slot;
  if (!work_item(a, b, s, g, empty_slot)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, qd = lane >> 4;
  const int h0 = g * HPG;
  const bool active = n < 2 * HPG;
  const bool is_lo = n >= HPG;
  const int col_head = !active ? 0 : (is_lo ? 2 * HPG - 1 - n : n);
  const bf16x8 zero8 = as_bf16x8(u32x4{0u, 0u, 0u, 0u});

  const int L = clamp_len(a.lens, b, a.t_max);
  int r0, r1;
  split_rows(L, a.S, a.split_rows, s, r0, r1);
  if (r0 >= r1 && s > 0) {                     // an empty split past the first: lse only
    if (tid < HPG) a.lse_part[((int64_t)b * a.H + h0 + tid) * a.S + s] = -INFINITY;
    return;
  }
  const int P = L - 1;                         // the query's position

  // ---- streaming setup (as in the GVA kernel: descriptors ending at the
  // split's last layout tile, zero reads past it); the first tiles are
  // requested before W is built
  const int r1c = ((r1 + kLayoutRows - 1) / kLayoutRows) * kLayoutRows;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + ((int64_t)b * a.G + g) * a.t_max * DV;
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(vbase), (short)0, r1c * DV * 2, kBufferWord3);
  const int v_lane = qd * 256 + n * 16;
  const int v_tile_bytes = 16 * DV * 2;
  const int ntiles = (r1 - r0 + TR - 1) / TR;
  const int my_tiles = ntiles > w ? (ntiles - w + kRopeWaves - 1) / kRopeWaves : 0;
  auto tile_row = [&](int j) { return r0 + (w + kRopeWaves * j) * TR; };
  struct VTile { bf16x8 v[HF][NC]; };
  // the 16-row blocks [hf0, hf1) of the tile at row0
  auto load_blocks = [&](VTile& t, int row0, int hf0, int hf1) {
    const int lt = row0 / kLayoutRows;
#pragma unroll
    for (int hf = hf0; hf < hf1; ++hf)
#pragma unroll
      for (int c = 0; c < NC; ++c)
        t.v[hf][c] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(vres, v_lane + 1024 * c, (lt + hf) * v_tile_bytes, kAuxNT));
  };
  VTile buf[DEPTH];
  if constexpr (DEPTH == 1) {
    load_blocks(buf[0], tile_row(0), 0, HF);
  } else {
#pragma unroll
    for (int d = 0; d < DEPTH - 1; ++d) load_blocks(buf[d], tile_row(d), 0, HF);
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- W_h for the group's heads, in LDS as 16-byte pieces:
  // piece ((hl * NC + kc) * NBC + nb) * 64 + (16 qd + n) holds
  // W[32 kc + 8 qd + j][16 nb + n], j = 0..7 -- the MFMA A operand of
  // W^T.  One task = 8 rows x one column pair of one head; consecutive
  // threads take consecutive pairs, so each row of M_h is read in whole
  // 4-byte pairs by neighbouring lanes.
  {
    u32x4* wl = reinterpret_cast<u32x4*>(lds);
    constexpr int PAIRS = DC / 2, RB = DV / 8;
    constexpr int TASKS = HPG * RB * PAIRS;
    for (int task = tid; task < TASKS; task += kRopeThreads) {
      const int i = task % PAIRS, rb = (task / PAIRS) % RB, hl = task / (PAIRS * RB);
      const int h = h0 + hl;
      const uint32_t qb = *reinterpret_cast<const uint32_t*>(
          static_cast<const uint16_t*>(a.q) + ((int64_t)b * a.H + h) * DC + 2 * i);
      const uint16_t* mrow = static_cast<const uint16_t*>(a.m) + ((int64_t)h * DV + 8 * rb) * DC + 2 * i;
      uint32_t mb[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) mb[j] = *reinterpret_cast<const uint32_t*>(mrow + (int64_t)j * DC);
      const float q0 = bf16_bits_to_f32(qb & 0xFFFFu) * a.scale_log2;
      const float q1 = bf16_bits_to_f32(qb >> 16) * a.scale_log2;
      float we[8], wo[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float m0 = bf16_bits_to_f32(mb[j] & 0xFFFFu), m1 = bf16_bits_to_f32(mb[j] >> 16);
        we[j] = q0 * m0 + q1 * m1;
        wo[j] = q1 * m0 - q0 * m1;
      }
      const int kc = rb >> 2, pqd = rb & 3, nb = i >> 3, pn = 2 * (i & 7);
      u32x4* dst = wl + ((hl * NC + kc) * NBC + nb) * 64 + 16 * pqd + pn;
      dst[0] = __builtin_bit_cast(u32x4, split_hi_lo(we, false));
      dst[1] = __builtin_bit_cast(u32x4, split_hi_lo(wo, false));
    }
    // angles of each wave's first tile, reduced exactly in fp64, and the
    // per-tile step (the wave's tiles lie kRopeWaves * TR rows apart)
    auto turns_u32 = [](double r) {
      return (uint32_t)(unsigned long long)((r - floor(r)) * 4294967296.0);
    };
    for (int i = tid; i < kRopeWaves * (DC / 2); i += kRopeThreads) {
      const int ww = i / (DC / 2), pi = i % (DC / 2);
      ang_all[i] = turns_u32(p.freq_rev[pi] * (double)(r0 + TR * ww - P));
    }
    for (int i = tid; i < DC / 2; i += kRopeThreads) {
      ang_step[i] = turns_u32(p.freq_rev[i] * (double)(TR * kRopeWaves));
      freq_f[i] = (float)p.freq_rev[i];
    }
  }
  __syncthreads();                              // W and the frequencies are in LDS

  bf16x8 esel[2];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    u32x4 u = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (8 * qd + j == n + 16 * half) u[j >> 1] |= 0x3F80u << (16 * (j & 1));
    esel[half] = as_bf16x8(u);
  }
  const u32x4* wl = reinterpret_cast<const u32x4*>(lds);
  float* xs = xs_all + w * HPG * TR;             // this wave's score transpose: [HPG][TR rows]

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[NB];
#pragma unroll
  for (int ib = 0; ib < NB; ++ib) acc[ib] = f32x4{0.f, 0.f, 0.f, 0.f};

  // next_row: with one tile in flight, the tile whose blocks are requested
  // as soon as the P.V has read this tile's (the registers are reused)
  auto compute_tile = [&](VTile& t, int row0, int row_end, int next_row) {
    if (row0 + TR > row_end) {
#pragma unroll
      for (int hf = 0; hf < HF; ++hf) {
        const bool dead = row0 + 16 * hf + n >= row_end;
#pragma unroll
        for (int c = 0; c < NC; ++c) t.v[hf][c] = dead ? zero8 : t.v[hf][c];
      }
    }
    // lane (n, qd): rows row0 + 16 hf + n, columns 16 nb + 4 qd + jj, i.e.
    // pairs i0 = 8 nb + 2 qd (jj = 0, 1) and i0 + 1 (jj = 2, 3)
    float sp[HPG][HF];
#pragma unroll
    for (int hl = 0; hl < HPG; ++hl)
#pragma unroll
      for (int hf = 0; hf < HF; ++hf) sp[hl][hf] = 0.f;
    // cos / sin of theta_i (t - P) for this lane's rows and the column
    // block's pairs: [hf][jj] = cos, sin, cos, sin.  The tile's first row
    // comes from the wave's 32-bit angle (exact to 2^-32 turns), the
    // lane's row offset within the tile (< TR rows) is added in fp32.
    const uint32_t* ang = ang_all + w * (DC / 2);
    // the wave's tile index: its tiles lie kRopeWaves tiles apart
    const uint32_t jt = (uint32_t)((row0 - r0) / (TR * kRopeWaves));
    auto trig = [&](int nb, float (&tr)[HF][4]) {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int pi = 8 * nb + 2 * qd + e;
        const uint32_t a = ang[pi] + jt * ang_step[pi];               // mod one turn
        const float rb = (float)a * 2.3283064365386963e-10f;          // 2^-32
        const float rc = rb + 0.25f;                                  // cos x = sin(x + 1/4 turn)
        const float ff = freq_f[pi];
#pragma unroll
        for (int hf = 0; hf < HF; ++hf) {
          const float dr = (float)(16 * hf + n);
          tr[hf][2 * e] = __builtin_amdgcn_sinf(fmaf(ff, dr, rc));
          tr[hf][2 * e + 1] = __builtin_amdgcn_sinf(fmaf(ff, dr, rb));
        }
      }
    };
    // Software pipeline over the (column block, head) steps: while the
    // matrix cores run one step's products, the LDS reads of the next
    // step's W piece and the cos/sin weighting of the previous step's
    // product issue (the order is pinned by scheduling barriers; left to
    // itself the compiler serialised read, products and weighting).  The
    // cos / sin of a column block are computed at its first step, after
    // the previous block's last weighting, into the same registers.
    constexpr int NIT = NBC * HPG;
    bf16x8 wa[2][NC];
    f32x4 gt[2][HF];
    float tr[HF][4];
    auto load_w = [&](int it, bf16x8 (&dst)[NC]) {
      const int nb = it / HPG, hl = it % HPG;
#pragma unroll
      for (int c = 0; c < NC; ++c) dst[c] = as_bf16x8(wl[((hl * NC + c) * NBC + nb) * 64 + lane]);
    };
    auto weight = [&](int it, const f32x4 (&g)[HF]) {
      const int hl = it % HPG;
#pragma unroll
      for (int hf = 0; hf < HF; ++hf)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) sp[hl][hf] = fmaf(g[hf][jj], tr[hf][jj], sp[hl][hf]);
    };
    auto products = [&](const bf16x8 (&wp)[NC], f32x4 (&g)[HF]) {
#pragma unroll
      for (int hf = 0; hf < HF; ++hf) g[hf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int hf = 0; hf < HF; ++hf) g[hf] = mfma16(wp[c], t.v[hf][c], g[hf]);
    };
    // (eight heads of 128-wide values leave no registers for the second
    // set of operands: those steps run in order)
    constexpr bool PIPE = !(HPG >= 8 && DV >= 128);
    if constexpr (!PIPE) {
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        if (it % HPG == 0) trig(it / HPG, tr);
        load_w(it, wa[0]);
        products(wa[0], gt[0]);
        weight(it, gt[0]);
      }
    } else {
      load_w(0, wa[0]);
      trig(0, tr);
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int cur = it & 1;
        products(wa[cur], gt[cur]);
        __builtin_amdgcn_sched_barrier(0);
        if (it + 1 < NIT) load_w(it + 1, wa[cur ^ 1]);
        if (it > 0) weight(it - 1, gt[cur ^ 1]);
        if (it > 0 && it % HPG == 0) trig(it / HPG, tr);
        __builtin_amdgcn_sched_barrier(0);
      }
      weight(NIT - 1, gt[(NIT - 1) & 1]);
    }
    // sum over the four 16-lane rows, then transpose through LDS: lane
    // (n, qd) takes head col_head's rows 32 rh + 16 k' + 4 qd + jj
#pragma unroll
    for (int hl = 0; hl < HPG; ++hl)
#pragma unroll
      for (int hf = 0; hf < HF; ++hf) xs[hl * TR + 16 * hf + n] = sum_over_rows(sp[hl][hf]);
    float x[RH][8];
#pragma unroll
    for (int rh = 0; rh < RH; ++rh) {
      const f32x4 lo = *reinterpret_cast<const f32x4*>(xs + col_head * TR + 32 * rh + 4 * qd);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(xs + col_head * TR + 32 * rh + 16 + 4 * qd);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        x[rh][jj] = lo[jj];
        x[rh][4 + jj] = hi[jj];
      }
    }
    if (row0 + TR > row_end) {
#pragma unroll
      for (int rh = 0; rh < RH; ++rh)
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (row0 + 32 * rh + 16 * (k >> 2) + 4 * qd + (k & 3) >= row_end) x[rh][k] = -INFINITY;
    }
    float mt = x[0][0];
#pragma unroll
    for (int rh = 0; rh < RH; ++rh)
#pragma unroll
      for (int k = 0; k < 8; ++k) mt = fmaxf(mt, x[rh][k]);
    mt = max_over_rows(mt);
    const float m_new = fmaxf(m_run, mt);
    if (__ballot(m_new > m_run) != 0) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) acc[ib] *= alpha;
      m_run = m_new;
    }
    float psum = 0.f;
    bf16x8 bp[RH];
#pragma unroll
    for (int rh = 0; rh < RH; ++rh) {
      float pr[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        pr[k] = __builtin_amdgcn_exp2f(x[rh][k] - m_run);
        psum += pr[k];
      }
      bp[rh] = active ? split_hi_lo(pr, is_lo) : zero8;
    }
    l_run += psum;
#pragma unroll
    for (int rh = 0; rh < RH; ++rh) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const f32x4 z = {0.f, 0.f, 0.f, 0.f};
          const f32x4 t0 = mfma16(t.v[2 * rh][c], esel[half], z);
          const f32x4 t1 = mfma16(t.v[2 * rh + 1][c], esel[half], z);
          bf16x8 av;
          const bf16x2 a01 = __builtin_convertvector((f32x2{t0[0], t0[1]}), bf16x2);
          const bf16x2 a23 = __builtin_convertvector((f32x2{t0[2], t0[3]}), bf16x2);
          const bf16x2 a45 = __builtin_convertvector((f32x2{t1[0], t1[1]}), bf16x2);
          const bf16x2 a67 = __builtin_convertvector((f32x2{t1[2], t1[3]}), bf16x2);
          av[0] = a01[0]; av[1] = a01[1]; av[2] = a23[0]; av[3] = a23[1];
          av[4] = a45[0]; av[5] = a45[1]; av[6] = a67[0]; av[7] = a67[1];
          acc[2 * c + half] = mfma16(av, bp[rh], acc[2 * c + half]);
        }
      if constexpr (DEPTH == 1) load_blocks(t, next_row, 2 * rh, 2 * rh + 2);
    }
  };

  if constexpr (DEPTH == 1) {
    for (int j = 0; j < my_tiles; ++j) compute_tile(buf[0], tile_row(j), r1, tile_row(j + 1));
  } else {
    for (int jt = 0; jt < my_tiles; jt += DEPTH) {
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        const int j = jt + d;
        if (j >= my_tiles) break;
        load_blocks(buf[(d + DEPTH - 1) % DEPTH], tile_row(j + DEPTH - 1), 0, HF);
        __builtin_amdgcn_sched_barrier(0);
        compute_tile(buf[d], tile_row(j), r1, 0);
      }
    }
  }

  // ---- merge the waves and write this split's partial
  l_run = sum_over_rows(l_run);
#pragma unroll
  for (int ib = 0; ib < NB; ++ib)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) acc[ib][jj] += mirror<HPG>(acc[ib][jj]);

  __syncthreads();   // W is dead: its LDS holds the per-wave records below
  constexpr int RS = DV + 2;
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
  for (int idx = tid; idx < HPG * DV; idx += kRopeThreads) {
    const int hl = idx / DV, i = idx % DV;
    float mx = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kRopeWaves; ++ww) mx = fmaxf(mx, red[(ww * HPG + hl) * RS]);
    float o = 0.f, lsum = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int ww = 0; ww < kRopeWaves; ++ww) {
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

using RopeDecodeFn = void (*)(RopeDecodeParams);

// W_h of every head of a group must fit the LDS budget of one workgroup.
template <int HPG, int DV, int DC>
RopeDecodeFn rope_if_fits() {
  if constexpr (HPG * DV * DC * 2 <= 128 * 1024) return rope_decode_kernel<HPG, DV, DC>;
  return nullptr;
}

template <int HPG, int DV>
RopeDecodeFn pick_rope_dc(int dc) {
  switch (dc) {
    case 64: return rope_if_fits<HPG, DV, 64>();
    case 128: return rope_if_fits<HPG, DV, 128>();
  }
  return nullptr;
}

template <int HPG>
RopeDecodeFn pick_rope_dv(int dv, int dc) {
  switch (dv) {
    case 64: return pick_rope_dc<HPG, 64>(dc);
    case 128: return pick_rope_dc<HPG, 128>(dc);
  }
  return nullptr;
}

RopeDecodeFn pick_rope_decode(int hpg, int dv, int dc) {
  switch (hpg) {
    case 1: return pick_rope_dv<1>(dv, dc);
    case 2: return pick_rope_dv<2>(dv, dc);
    case 4: return pick_rope_dv<4>(dv, dc);
    case 8: return pick_rope_dv<8>(dv, dc);
  }
  return nullptr;
}

// The absorption behind gva_absorb_query (one query row per sequence) and
// gva_prefill_absorb (a sequence's last n_per_seq rows).
}  // namespace

extern "C" {

int gva_rope_decode_attention(const gva_dims* dims, const void* q, const void* m, const void* v_cache,
                              const int32_t* lens, int32_t num_splits, int32_t split_rows, float* o_part,
                              float* lse_part, void* stream) {
  int st = check_dims(dims);
  if (st != GVA_OK) return st;
  if (dims->d_r != 0 || dims->d_c < 2 || (dims->d_c & 1)) return GVA_ERR_INVALID_ARG;
  if (!(dims->rope_base > 0.0) || !isfinite(dims->rope_base)) return GVA_ERR_INVALID_ARG;
  if (num_splits < 1 || num_splits > GVA_MAX_SPLITS) return GVA_ERR_INVALID_ARG;
  if (split_rows < 0 || split_rows % kTileRows != 0) return GVA_ERR_INVALID_ARG;
  if (!q || !m || !v_cache || !lens || !o_part || !lse_part) return GVA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(m, 16) || !aligned(v_cache, 16) || !aligned(lens, 4) ||
      !aligned(o_part, 16) || !aligned(lse_part, 4))
    return GVA_ERR_INVALID_ARG;
  if (dims->dtype != GVA_DTYPE_BF16) return GVA_ERR_UNSUPPORTED;
  st = check_cache_layout(dims);
  if (st != GVA_OK) return st;
  const int hpg = dims->n_heads / dims->n_groups;
  RopeDecodeFn fn = pick_rope_decode(hpg, dims->d_v, dims->d_c);
  if (fn == nullptr) return GVA_ERR_UNSUPPORTED;
  const long long n_items = decode_grid(dims, num_splits, split_rows);
  if (n_items > 0x7FFFFFFFLL) return GVA_ERR_UNSUPPORTED;

  RopeDecodeParams p{};
  memset(&p, 0, sizeof(p));
  p.a.q = q;
  p.a.m = m;
  p.a.v = const_cast<void*>(v_cache);       // read only
  p.a.lens = lens;
  p.a.o_part = o_part;
  p.a.lse_part = lse_part;
  p.a.B = dims->batch;
  p.a.H = dims->n_heads;
  p.a.G = dims->n_groups;
  p.a.d_v = dims->d_v;
  p.a.d_c = dims->d_c;
  p.a.d_r = 0;
  p.a.t_max = dims->t_max;
  p.a.S = num_splits;
  p.a.split_rows = split_rows;
  p.a.scale_log2 = scale_log2(dims);        // d_r = 0: 1/sqrt(d_c) unless given
  constexpr double kInv2Pi = 0.15915494309189533577;
  for (int i = 0; i < dims->d_c / 2; ++i)
    p.freq_rev[i] = pow(dims->rope_base, -2.0 * (double)i / (double)dims->d_c) * kInv2Pi;
  hipLaunchKernelGGL(fn, dim3((unsigned)n_items), dim3(kRopeThreads), 0, static_cast<hipStream_t>(stream), p);
  return launch_status();
}

}  // extern "C"
