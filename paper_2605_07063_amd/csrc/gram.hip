// Target mean, Gram matrix and alignment scores per parameter group (dr_gram).
//
// Per group p (a column range of the sketch matrix, Sec. 3.3.3):
//   gbar_p = mean of the m target rows            (Sec. 3.2)
//   K_p    = G_p G_p^T                             (redundancy term, Sec. 3.3.2)
//   s_p    = G_p gbar_p,  t2_p = ||gbar_p||^2      (alignment scores)
//
// Kernels
//   target_mean_kernel : gbar in fp32 (fp64 sum over the m rows).
//   gram_tile_kernel   : bf16 rows: one 64x64 tile of K_p over one chunk of
//                        the group's columns (lower-triangle tile pairs only),
//                        bf16 16x16x32 MFMA, fp32 accumulate; operands stream
//                        from memory straight into registers.
//   gram_tile_lds_kernel : fp32 rows, the same tiles and chunks on fp32
//                        16x16x4 MFMA, the workgroup's rows staged once per
//                        step through a three-stage LDS ring.  A diagonal
//                        tile stages its rows once plus the target mean, and
//                        its wave above the diagonal forms s_p for the
//                        tile's rows (tile 0 also t2_p), so the same pass
//                        yields them.
//   gram_reduce_kernel : sums the chunk partials of a tile in chunk order and
//                        writes the lower triangle and its mirror, so K is
//                        exactly symmetric, and for fp32 sketches s_p and
//                        t2_p from the diagonal tiles.
//   score_kernel       : s_p[i] = <G_p[i], gbar_p> and t2_p against the fp32
//                        mean, fp64 accumulation, fixed-order block
//                        reduction: bf16 sketches, and t2_p of fp32 ones
//                        with n = 0.
// Large bf16 problems (at least kBigMinTiles 256x256 lower-triangle tiles):
//   gram_big_kernel    : one 256x256 tile of K_p per workgroup over all of
//                        the group's columns (no split): 64-column steps
//                        stream into a two-stage LDS ring by buffer->LDS DMA,
//                        four waves (one per SIMD) each hold a 128x128 fp32
//                        accumulator in AGPRs (bf16 16x16x32 MFMA); lower-
//                        triangle tiles only, scheduled in 4x8-tile chunks,
//                        one per XCD at a time.  Each tile goes out from
//                        registers in non-temporal float4 stores, also
//                        transposed into the upper triangle, so K is exactly
//                        symmetric without a second pass.
// Small fp32 problems (n + 1 <= 128 rows: the per-step batches):
//   gram_small_kernel  : one workgroup per 128-column chunk of a group forms
//                        the chunk of gbar from the target rows (fp64 sum /
//                        m, as target_mean_kernel) and stages the n + 1
//                        augmented rows in LDS (row stride 132 floats: the
//                        16 rows x 4 columns of an fp32 MFMA operand fall on
//                        distinct banks); the eight waves take the lower
//                        16x16 blocks of the augmented Gram round-robin
//                        (fp32 16x16x4 MFMA) and write chunk partials.
//   gram_small_reduce_kernel : sums the chunk partials (one wave per element,
//                        a fixed order) into K (both triangles), s (row n)
//                        and t2 (element n, n).
// No atomics: results are deterministic.

#include <mutex>
#include <type_traits>

#include "common.h"

namespace dr {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;
constexpr int kMaxGroups = 256;   // groups per launch (more groups -> more launches)
constexpr int kTargetWGs = 1024;
constexpr int kLdsSlots = 256 * 3;   // gram_tile_lds_kernel workgroups resident at once: 256 CUs x 3 (48 KB of LDS each)

struct GramArgs {
  const unsigned char* G;
  long long ldG;
  int n;
  int rows;                         // rows of the Gram problem: n, or n + 1 with gbar as row n
  const float* gbar;                // [cols] by absolute column (row n when rows == n + 1)
  long long goff[kMaxGroups + 1];   // absolute column offsets of this launch's groups
  int P;
  int NT, pairs, CK, maxchunks;
  float* partial;                   // [P][pairs][maxchunks][kTile*kTile]
  float* K;                         // outputs (gram_tile_lds_kernel writes them itself when
  float* s;                         // maxchunks == 1); group p of the launch is pbase + p
  float* t2;
  long long pbase;
};

template <bool BF16>
struct GTr;
template <>
struct GTr<true> {
  static constexpr int ES = 2, EPV = 8, KV = 32;   // KV: columns per 16-byte vector per lane group
};
template <>
struct GTr<false> {
  static constexpr int ES = 4, EPV = 4, KV = 16;
};

template <bool BF16>
__device__ __forceinline__ f32x4 mma_v(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (BF16) {
    return mma_bf16(a, b, c);
  } else {
    c = mma_f32(__uint_as_float(a.x), __uint_as_float(b.x), c);
    c = mma_f32(__uint_as_float(a.y), __uint_as_float(b.y), c);
    c = mma_f32(__uint_as_float(a.z), __uint_as_float(b.z), c);
    c = mma_f32(__uint_as_float(a.w), __uint_as_float(b.w), c);
    return c;
  }
}

__device__ __forceinline__ void pair_to_tiles(int q, int& I, int& J) {
  int i = (int)((sqrtf(8.f * q + 1.f) - 1.f) * 0.5f);
  while ((i + 1) * (i + 2) / 2 <= q) ++i;
  while (i * (i + 1) / 2 > q) --i;
  I = i;
  J = q - i * (i + 1) / 2;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads, 2) void gram_tile_kernel(GramArgs a) {
  using E = GTr<BF16>;
  constexpr int NV = 2;              // vectors per row-block per step
  constexpr int STEP = NV * 4 * E::EPV;   // columns per step (4 lane groups)
  const int chunk = blockIdx.x, q = blockIdx.y, p = blockIdx.z;
  const long long g0 = a.goff[p], g1 = a.goff[p + 1];
  const long long c0 = g0 + (long long)chunk * a.CK;
  if (c0 >= g1) return;
  const long long c1 = c0 + a.CK < g1 ? c0 + a.CK : g1;
  int I, J;
  pair_to_tiles(q, I, J);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wr = wave >> 1, wc = wave & 1;

  int rowA[2], rowB[2];
  bool okA[2], okB[2];
  const unsigned char* baseA[2];
  const unsigned char* baseB[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    rowA[b] = I * kTile + wr * 32 + b * 16 + lr;
    rowB[b] = J * kTile + wc * 32 + b * 16 + lr;
    okA[b] = rowA[b] < a.rows;
    okB[b] = rowB[b] < a.rows;
    // row n of the augmented problem is the fp32 target mean (fp32 path only)
    baseA[b] = rowA[b] < a.n ? a.G + (long long)rowA[b] * a.ldG * E::ES
                             : reinterpret_cast<const unsigned char*>(a.gbar);
    baseB[b] = rowB[b] < a.n ? a.G + (long long)rowB[b] * a.ldG * E::ES
                             : reinterpret_cast<const unsigned char*>(a.gbar);
  }

  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](long long cs, u32x4 (&va)[2][NV], u32x4 (&vb)[2][NV]) {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const long long c = cs + (long long)v * 4 * E::EPV + lg * E::EPV;
      const bool cok = c < c1;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        // unconditional loads (an entry outside the problem reads the first
        // 16 bytes of the target mean instead, which every call has: G may
        // be empty, and then null; the value is then zeroed), so that the
        // compiler's waits count the loads in flight
        const unsigned char* dummy = reinterpret_cast<const unsigned char*>(a.gbar);
        const bool ea = okA[b] && cok, eb = okB[b] && cok;
        const u32x4 xa = *reinterpret_cast<const u32x4*>(ea ? baseA[b] + c * E::ES : dummy);
        const u32x4 xb = *reinterpret_cast<const u32x4*>(eb ? baseB[b] + c * E::ES : dummy);
        va[b][v] = ea ? xa : u32x4{0u, 0u, 0u, 0u};
        vb[b][v] = eb ? xb : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };

  // DEPTH steps of loads in flight: the operands come from L2 straight
  // into registers, so their latency is what the products wait for; loads
  // past the chunk read zeros (no memory access), whose products add 0
  constexpr int DEPTH = 3;
  u32x4 ba[DEPTH][2][NV], bb[DEPTH][2][NV];
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d) load(c0 + (long long)d * STEP, ba[d], bb[d]);
  for (long long cs = c0; cs < c1; cs += DEPTH * STEP) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      load(cs + (long long)(d + DEPTH - 1) * STEP, ba[(d + DEPTH - 1) % DEPTH], bb[(d + DEPTH - 1) % DEPTH]);
      // the loads go out before this step's products (the scheduler would
      // otherwise move them next to their uses)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mma_v<BF16>(ba[d][i][v], bb[d][j][v], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  float* out = a.partial + (((long long)p * a.pairs + q) * a.maxchunks + chunk) * (kTile * kTile);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        out[(wr * 32 + i * 16 + lg * 4 + r) * kTile + wc * 32 + j * 16 + lr] = acc[i][j][r];
}


// fp32 rows, n + 1 > 128: 64 x 64 tile pairs over the n general rows, with
// the operands staged through LDS.  Per step of 32 columns the workgroup's
// rows are loaded once into registers (16-byte segments), written to a
// three-stage LDS ring in the conflict-free operand layout, and read by the
// four waves as fp32 MFMA fragments; loads run two steps ahead of their LDS
// writes, and the LDS writes one step ahead of the products.
//   off-diagonal pair (I > J): tile I's 64 rows, then tile J's 64 rows;
//   diagonal pair (I = J): tile I's 64 rows once (they are both operands),
//     then the target mean as a 16-row block whose other rows are zero.
//     Waves (0, 0), (1, 0) and (1, 1) take the tile's lower triangle; wave
//     (0, 1), whose quadrant lies above the diagonal, takes the target mean
//     against the 64 rows (the scores s), and in tile 0 wave (0, 0) also
//     takes the target mean against itself (t2).  Both land in the partial
//     tile's upper triangle, which holds nothing else: s of tile row
//     16 b + l at (16 (b / 2), 32 + 16 (b % 2) + l), t2 at (0, 16).
constexpr int kLS = 32;                          // fp32 columns per step (128-byte rows)
constexpr int kLNS = 3;                          // ring stages
constexpr int kLStage = 2 * kTile * kLS * 4;     // 128 rows of 128 bytes
constexpr int kLMeanRow = kTile;                 // diagonal pairs: the target mean's stage row
constexpr int kKindS = 16, kKindT2 = 17;         // wave tasks beyond the block masks 0..15

__global__ __launch_bounds__(kThreads, 2) void gram_tile_lds_kernel(GramArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLNS * kLStage];
  const int chunk = blockIdx.x, q = blockIdx.y, p = blockIdx.z;
  const long long g0 = a.goff[p], g1 = a.goff[p + 1];
  const long long c0 = g0 + (long long)chunk * a.CK;
  // with one chunk per group the tile is final and written here, so an
  // empty group still writes its zeros (no steps)
  const bool direct = a.maxchunks == 1;
  if (c0 >= g1 && !direct) return;
  const long long c1 = c0 + a.CK < g1 ? c0 + a.CK : g1;
  const int nsteps = c1 > c0 ? (int)((c1 - c0 + kLS - 1) / kLS) : 0;
  int I, J;
  pair_to_tiles(q, I, J);
  const bool diag = I == J;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wr = w >> 1, wc = w & 1;
  // loader: segment e = tid + 256 u of a stage is stage row e / 8, segment
  // e % 8 (an off-diagonal pair loads u = 0..3, a diagonal one u = 0..2).
  // An entry outside the problem reads the target mean's first 16 bytes
  // instead and is zeroed at the LDS write, so the loads are unconditional
  // and their waits counted.
  const unsigned char* mean = reinterpret_cast<const unsigned char*>(a.gbar);   // by absolute column
  const unsigned char* src[4];
  bool rok[4];
  int sseg[4];
  unsigned loff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid + kThreads * u, R = e >> 3, sg = e & 7;
    if (R < kTile || !diag) {
      const int grow = R < kTile ? I * kTile + R : J * kTile + (R - kTile);
      rok[u] = grow < a.n;
      src[u] = rok[u] ? a.G + (long long)grow * a.ldG * 4 : mean;
    } else {
      rok[u] = R == kLMeanRow;
      src[u] = mean;
    }
    sseg[u] = sg;
    loff[u] = (unsigned)(R * 128 + ((sg ^ ((R >> 1) & 7)) * 16));
  }
  auto seg_ok = [&](int t, int u) { return rok[u] && c0 + (long long)t * kLS + sseg[u] * 4 < c1; };
  // the zeroing happens at the LDS write, so nothing waits for the loads
  // until then
  auto gload = [&](int t, u32x4 (&v)[4], auto nu) {
#pragma unroll
    for (int u = 0; u < decltype(nu)::value; ++u) {
      const long long c = c0 + (long long)t * kLS + sseg[u] * 4;
      v[u] = *reinterpret_cast<const u32x4*>(seg_ok(t, u) ? src[u] + c * 4 : mean);
    }
  };
  auto lstore = [&](int t, const u32x4 (&v)[4], auto nu) {
    unsigned char* sb = lds + (t % kLNS) * kLStage;
#pragma unroll
    for (int u = 0; u < decltype(nu)::value; ++u)
      *reinterpret_cast<u32x4*>(sb + loff[u]) = seg_ok(t, u) ? v[u] : u32x4{0u, 0u, 0u, 0u};
  };
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the wave's products of step t.  Kind 0..15: the 16 x 16 blocks (i, j)
  // whose bit i * 2 + j is set (A block i against B block j); kKindT2: mask
  // 13 plus the target mean against itself into acc[0][1]; kKindS: the
  // target mean against the tile's four 16-row blocks into acc[b / 2][b % 2]
  auto compute = [&](int t, auto kind, auto dg) {
    constexpr int KD = decltype(kind)::value;
    constexpr bool DG = decltype(dg)::value;
    if constexpr (KD != 0) {
      const unsigned char* sb = lds + (t % kLNS) * kLStage;
      const unsigned char* bb = sb + (DG ? 0 : kTile * 128);   // B operand rows
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        const int sg = 4 * kh + lg;
        if constexpr (KD == kKindS) {
          const u32x4 fm = swz_read(sb + kLMeanRow * 128, lr, sg);
          u32x4 fb[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) fb[b] = swz_read(sb + 16 * b * 128, lr, sg);
          acc[0][0] = mma_v<false>(fm, fb[0], acc[0][0]);
          acc[0][1] = mma_v<false>(fm, fb[1], acc[0][1]);
          acc[1][0] = mma_v<false>(fm, fb[2], acc[1][0]);
          acc[1][1] = mma_v<false>(fm, fb[3], acc[1][1]);
        } else {
          constexpr int M = KD == kKindT2 ? 13 : KD;
          constexpr bool ra0 = (M & 3) != 0, ra1 = (M & 12) != 0, rb0 = (M & 5) != 0, rb1 = (M & 10) != 0;
          u32x4 fa[2], fb[2];
          if constexpr (ra0) fa[0] = swz_read(sb + (wr * 32) * 128, lr, sg);
          if constexpr (ra1) fa[1] = swz_read(sb + (wr * 32 + 16) * 128, lr, sg);
          if constexpr (rb0) fb[0] = swz_read(bb + (wc * 32) * 128, lr, sg);
          if constexpr (rb1) fb[1] = swz_read(bb + (wc * 32 + 16) * 128, lr, sg);
          if constexpr ((M & 1) != 0) acc[0][0] = mma_v<false>(fa[0], fb[0], acc[0][0]);
          if constexpr ((M & 2) != 0) acc[0][1] = mma_v<false>(fa[0], fb[1], acc[0][1]);
          if constexpr ((M & 4) != 0) acc[1][0] = mma_v<false>(fa[1], fb[0], acc[1][0]);
          if constexpr ((M & 8) != 0) acc[1][1] = mma_v<false>(fa[1], fb[1], acc[1][1]);
          if constexpr (KD == kKindT2) {
            const u32x4 fm = swz_read(sb + kLMeanRow * 128, lr, sg);
            acc[0][1] = mma_v<false>(fm, fm, acc[0][1]);
          }
        }
      }
    }
  };
  // step t: products from stage t % 3; the data of step t + 2 (loaded two
  // steps ago) into stage (t + 2) % 3, last read at step t - 1; the loads of
  // step t + 4; one barrier
  auto run = [&](auto dg, auto kind) {
    constexpr bool DG = decltype(dg)::value;
    const std::integral_constant<int, DG ? 3 : 4> nu;
    u32x4 va[4], vb[4];
    gload(0, va, nu);
    gload(1, vb, nu);
    lstore(0, va, nu);
    lstore(1, vb, nu);
    gload(2, va, nu);
    gload(3, vb, nu);
    __syncthreads();
    for (int t = 0; t < nsteps; t += 2) {
      compute(t, kind, dg);
      lstore(t + 2, va, nu);
      __builtin_amdgcn_sched_barrier(0);
      gload(t + 4, va, nu);
      __builtin_amdgcn_sched_barrier(0);
      DR_LDS_SYNC();
      compute(t + 1, kind, dg);   // past the last step its stage holds zeros: the products add 0
      lstore(t + 3, vb, nu);
      __builtin_amdgcn_sched_barrier(0);
      gload(t + 5, vb, nu);
      __builtin_amdgcn_sched_barrier(0);
      DR_LDS_SYNC();
    }
  };
  // Blocks the reduction never reads take no products and keep zero
  // accumulators: A rows wholly past row n - 1 (I >= J, so these are the
  // last tile's), and on a diagonal tile the blocks wholly above the
  // diagonal.  The mask is uniform over the wave and is rounded up to the
  // smallest loop variant that contains it (extra products are harmless).
  int live = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int rb = I * kTile + wr * 32 + 16 * i, cb = J * kTile + wc * 32 + 16 * j;
      if (rb < a.n && cb <= rb + 15) live |= 1 << (i * 2 + j);
    }
  using F = std::false_type;
  using T = std::true_type;
  if (!diag) {
    // J < I: every B block lies below the A rows, so live is 0, 3 or 15
    if (live == 0)
      run(F{}, std::integral_constant<int, 0>{});
    else if ((live & ~3) == 0)
      run(F{}, std::integral_constant<int, 3>{});
    else
      run(F{}, std::integral_constant<int, 15>{});
  } else if (wr == 0 && wc == 1) {
    run(T{}, std::integral_constant<int, kKindS>{});
  } else if (I == 0 && wr == 0 && wc == 0) {
    run(T{}, std::integral_constant<int, kKindT2>{});   // its live blocks are within mask 13
  } else if (live == 0) {
    run(T{}, std::integral_constant<int, 0>{});
  } else if ((live & ~1) == 0) {
    run(T{}, std::integral_constant<int, 1>{});
  } else if ((live & ~3) == 0) {
    run(T{}, std::integral_constant<int, 3>{});
  } else if ((live & ~13) == 0) {
    run(T{}, std::integral_constant<int, 13>{});
  } else {
    run(T{}, std::integral_constant<int, 15>{});
  }

  if (direct) {
    // the reduction's writes for a single chunk: K's lower triangle and
    // mirror, and from a diagonal tile the scores and t2 in its upper
    // triangle
    float* Kp = a.K + (a.pbase + p) * (long long)a.n * a.n;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tr = wr * 32 + i * 16 + lg * 4 + r, tc = wc * 32 + j * 16 + lr;
          const int row = I * kTile + tr, col = J * kTile + tc;
          const float v = acc[i][j][r];
          if (col <= row) {
            if (row < a.n) {
              Kp[(long long)row * a.n + col] = v;
              Kp[(long long)col * a.n + row] = v;
            }
          } else if (diag) {
            if ((tr == 0 || tr == 16) && tc >= 32) {
              const int srow = I * kTile + 2 * tr + (tc - 32);
              if (srow < a.n) a.s[(a.pbase + p) * (long long)a.n + srow] = v;
            } else if (I == 0 && tr == 0 && tc == 16) {
              a.t2[a.pbase + p] = v;
            }
          }
        }
    return;
  }
  float* out = a.partial + (((long long)p * a.pairs + q) * a.maxchunks + chunk) * (kTile * kTile);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        out[(wr * 32 + i * 16 + lg * 4 + r) * kTile + wc * 32 + j * 16 + lr] = acc[i][j][r];
}

// ---------------------------------------------------------------- small fp32

constexpr int kSmCK = 128;           // columns per workgroup
constexpr int kSmLd = kSmCK + 4;     // LDS row stride (floats)
constexpr int kSmMaxRows = 128;      // n + 1 <= 128
constexpr int kSmThreads = 512;      // eight waves share the lower blocks

__global__ __launch_bounds__(kSmThreads) void gram_small_kernel(GramArgs a, const float* Gt, long long ldGt, int m,
                                                              int NRP, int nchunks) {
  __shared__ __attribute__((aligned(16))) float R[kSmMaxRows * kSmLd];
  const int chunk = blockIdx.x, p = blockIdx.y;
  const long long g0 = a.goff[p], g1 = a.goff[p + 1];
  const long long c0 = g0 + (long long)chunk * kSmCK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nb = NRP / 16;
  float* out = a.partial + ((long long)p * nchunks + chunk) * NRP * NRP;
  if (c0 >= g1) return;   // (uniform) past the group: the reduction skips this chunk
  const int width = (int)(g1 - c0 < kSmCK ? g1 - c0 : kSmCK);   // a multiple of 4
  // general rows 0 .. n-1 (float4 loads, eight in flight per thread before
  // any store), zero columns past the group
  constexpr int RPP = kSmThreads / (kSmCK / 4);                    // rows per pass
  const int c4 = tid & (kSmCK / 4 - 1), r0 = tid / (kSmCK / 4);
  const bool cok = 4 * c4 < width;
  for (int rb = 0; rb < a.n; rb += 8 * RPP) {
    float4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int r = rb + r0 + RPP * u;
      v[u] = (r < a.n && cok) ? *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(a.G) +
                                                                 (long long)r * a.ldG + c0 + 4 * c4)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int r = rb + r0 + RPP * u;
      if (r < a.n) *reinterpret_cast<float4*>(&R[r * kSmLd + 4 * c4]) = v[u];
    }
  }
  // row n: the target mean of this chunk (fp64 sum over the m rows in order,
  // eight loads in flight); rows n + 1 .. NRP - 1: zeros
  if (tid < kSmCK) {
    float gv = 0.f;
    if (tid < width) {
      double acc = 0.0;
      for (int j0 = 0; j0 < m; j0 += 8) {
        float t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = j0 + u < m ? Gt[(long long)(j0 + u) * ldGt + c0 + tid] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (j0 + u < m) acc += (double)t[u];
      }
      gv = (float)(acc / (double)m);
    }
    R[a.n * kSmLd + tid] = gv;
  }
  for (int e = tid; e < (NRP - a.n - 1) * kSmCK; e += kSmThreads)
    R[(a.n + 1 + e / kSmCK) * kSmLd + e % kSmCK] = 0.f;
  __syncthreads();
  // lower blocks (I, J <= I) round-robin over the waves
  const int lr = lane & 15, lk = lane >> 4, lg = lane >> 4;
  const int nblocks = nb * (nb + 1) / 2;
  for (int q = wave; q < nblocks; q += kSmThreads / 64) {
    int I = 0;
    while ((I + 1) * (I + 2) / 2 <= q) ++I;
    const int J = q - I * (I + 1) / 2;
    const float* ra = &R[(16 * I + lr) * kSmLd + lk];
    const float* rb = &R[(16 * J + lr) * kSmLd + lk];
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int k = 0; k < kSmCK; k += 4) acc = mma_f32(ra[k], rb[k], acc);
    // C layout: register r is row 4 lg + r of the block, column lane % 16
#pragma unroll
    for (int r = 0; r < 4; ++r) out[(16 * I + 4 * lg + r) * NRP + 16 * J + lr] = acc[r];
  }
}

// K (both triangles), s and t2 from the chunk partials: one wave per element
// of the lower triangle, lane l sums chunks l, l + 64, ... in order, then a
// fixed-order DPP reduction across the lanes (total in lane 63)
__global__ __launch_bounds__(kThreads) void gram_small_reduce_kernel(GramArgs a, int NRP, int nchunks, float* K,
                                                                     float* s, float* t2, long long pbase) {
  const int p = blockIdx.y;
  const int nr = a.n + 1;
  const int e = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);   // lower-triangle element
  const int lane = threadIdx.x & 63;
  if (e >= nr * (nr + 1) / 2) return;
  int r = 0;
  while ((r + 1) * (r + 2) / 2 <= e) ++r;
  const int c = e - r * (r + 1) / 2;
  const long long width = a.goff[p + 1] - a.goff[p];
  const int nvalid = (int)((width + kSmCK - 1) / kSmCK);
  const float* src = a.partial + (long long)p * nchunks * NRP * NRP + r * NRP + c;
  float acc = 0.f;
  for (int ch0 = 0; ch0 < nvalid; ch0 += 256) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ch = ch0 + lane + 64 * u;
      v[u] = ch < nvalid ? src[(long long)ch * NRP * NRP] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) acc += v[u];
  }
  acc = wave_sum_l63f(acc);
  if (lane != 63) return;
  if (r < a.n) {
    float* Kp = K + (pbase + p) * (long long)a.n * a.n;
    Kp[(long long)r * a.n + c] = acc;
    Kp[(long long)c * a.n + r] = acc;
  } else if (c < a.n) {
    s[(pbase + p) * (long long)a.n + c] = acc;
  } else {
    t2[pbase + p] = acc;
  }
}

// ---------------------------------------------------------------- large n

constexpr int kBT = 256;                   // output tile edge
constexpr int kBK = 64;                    // bf16 columns per step (128-byte rows)
constexpr int kBPanel = kBT * kBK * 2;     // bytes of one operand panel per step (32 KiB)
constexpr int kBStage = 2 * kBPanel;       // A and B panels
constexpr int kBigMinTiles = 512;

struct BigArgs {
  const unsigned char* G;
  long long ldG;   // elements
  int n, T, pairs;
  int vec4;        // K rows start 16-byte aligned (n % 4 == 0, K aligned): float4 stores
  long long goff[kMaxGroups + 1];
  float* K;        // [P][n][n] of this launch's groups
};

// One 16x16 block of C (lane l holds C[4 (l / 16) + r][l % 16] in element r)
// into K at rows R.., columns C.. and, mirrored, at rows C.., columns R..,
// for an off-diagonal tile inside K with 16-byte aligned rows: every element
// goes out in non-temporal float4 stores.  The mirror is the accumulator as
// it stands (four consecutive rows of one column are four consecutive
// columns of the transposed row); the block itself after a 4 x 4 transpose
// inside each quad of lanes (two rounds of DPP quad permutations).
__device__ __forceinline__ void big_store_block_fast(float* Kp, int n, int R, int C, f32x4 v, int lane) {
  const int lr = lane & 15, lg = lane >> 4, c = lane & 3, m = lr >> 2;
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(Kp + (long long)(C + lr) * n + R + 4 * lg));
  float x0 = v[0], x1 = v[1], x2 = v[2], x3 = v[3];
  {  // exchange across bit 0 of the quad lane
    const float s01 = (c & 1) ? x0 : x1, s23 = (c & 1) ? x2 : x3;
    const float r01 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s01), 0xB1, 0xF, 0xF, false));
    const float r23 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s23), 0xB1, 0xF, 0xF, false));
    if (c & 1) { x0 = r01; x2 = r23; } else { x1 = r01; x3 = r23; }
  }
  {  // exchange across bit 1
    const float s02 = (c & 2) ? x0 : x2, s13 = (c & 2) ? x1 : x3;
    const float r02 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s02), 0x4E, 0xF, 0xF, false));
    const float r13 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s13), 0x4E, 0xF, 0xF, false));
    if (c & 2) { x0 = r02; x1 = r13; } else { x2 = r02; x3 = r13; }
  }
  __builtin_nontemporal_store(f32x4{x0, x1, x2, x3}, reinterpret_cast<f32x4*>(Kp + (long long)(R + 4 * lg + c) * n + C + 4 * m));
}

// the same block element by element: rows and columns past n are skipped,
// and in a diagonal tile only the lower triangle (with its mirror above)
__device__ __forceinline__ void big_store_block_masked(float* Kp, int n, bool diag, int R, int C, f32x4 v, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = R + 4 * lg + r, col = C + lr;
    if (row < n && col < n) {
      if (!diag || col <= row) Kp[(long long)row * n + col] = v[r];
      if (!diag || col < row) Kp[(long long)col * n + row] = v[r];
    }
  }
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gram_big_kernel(BigArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * kBStage];
  const int p = blockIdx.y;
  // Workgroup i runs on XCD i % 8, and an XCD's 32 CUs take its workgroups
  // in order.  The lower-triangle tiles are grouped in chunks of 4 tile rows
  // x 8 tile columns (bands of 4 rows, 8 columns at a time); XCD x runs
  // chunks x, x + 8, ... one whole chunk at a time, so the 32 concurrent
  // tiles of an XCD read 12 distinct panels through its L2 rather than ~34.
  int I, J;
  {
    const int x = blockIdx.x & 7, sl = blockIdx.x >> 3;
    const int ci = (sl >> 5) * 8 + x, r = sl & 31;
    int band = 0, acc = 0;
    for (;; ++band) {
      if (4 * band >= a.T) return;   // past the last chunk
      const int rows_end = 4 * band + 4 < a.T ? 4 * band + 4 : a.T;
      const int nc = (rows_end + 7) / 8;
      if (ci < acc + nc) break;
      acc += nc;
    }
    I = 4 * band + (r >> 3);
    J = 8 * (ci - acc) + (r & 7);
    if (I >= a.T || J > I) return;
  }
  const long long g0 = a.goff[p], g1 = a.goff[p + 1];
  const int nk = (int)((g1 - g0 + kBK - 1) / kBK);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w >> 1, wc = w & 1;   // 128-row half of A, 128-row half of B
  const int lr = lane & 15, lg = lane >> 4;
  const int rowA0 = I * kBT, rowB0 = J * kBT;
  const int rowsA = a.n - rowA0 < kBT ? a.n - rowA0 : kBT;
  const int rowsB = a.n - rowB0 < kBT ? a.n - rowB0 : kBT;
  const bool diag = I == J;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(a.G + (long long)rowA0 * a.ldG * 2, kOobOffset);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.G + (long long)rowB0 * a.ldG * 2, kOobOffset);
  // this lane's 8 rows of each panel (half blocks w, w + 4, ..., w + 28) and its segment
  unsigned offA[8], offB[8];
  int segs[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int hb = w + 4 * u;             // half block: rows 8 hb .. 8 hb + 7
    const int r = 8 * hb + (lane >> 3);
    segs[u] = swz_seg_of_lane(lane, hb & 1);
    offA[u] = r < rowsA ? (unsigned)((long long)r * a.ldG * 2) : kOobOffset;
    offB[u] = r < rowsB ? (unsigned)((long long)r * a.ldG * 2) : kOobOffset;
  }
  // DMA q (0..15) of step t into stage st: q even A, q odd B, half block
  // w + 4 (q / 2); steps past the group load zeros (no memory access)
  auto dma1 = [&](int t, int st, int q) {
    unsigned char* sb = lds + st * kBStage;
    const int u = q >> 1;
    const long long col = g0 + (long long)t * kBK + segs[u] * 8;
    const bool cok = col < g1;
    if (q & 1) {
      const unsigned cb = (offB[u] == kOobOffset || !cok) ? kOobOffset : offB[u] + (unsigned)(col * 2);
      dma16<kAuxCached>(rb, sb + kBPanel + (w + 4 * u) * 1024, cb);
    } else {
      const unsigned ca = (offA[u] == kOobOffset || !cok) ? kOobOffset : offA[u] + (unsigned)(col * 2);
      dma16<kAuxCached>(ra, sb + (w + 4 * u) * 1024, ca);
    }
  };
  // fragment read q (0..15) of 32-column half kh: q even A block q / 2, odd B block
  auto rd1 = [&](u32x4* fa, u32x4* fb, const unsigned char* sa, int kh, int q) {
    const int seg = 4 * kh + lg;
    if (q & 1) fb[q >> 1] = swz_read(sa + kBPanel + (wc * 8 + (q >> 1)) * 2048, lr, seg);
    else fa[q >> 1] = swz_read(sa + (wr * 8 + (q >> 1)) * 2048, lr, seg);
  };
  // The 128 x 128 accumulator (256 registers) sits in the AGPRs: each product
  // is an in-place asm MFMA on its accumulator, so the register allocator
  // keeps every accumulator where it is (the compiler's own MFMA form moves
  // them between register files at this size).  Volatile asm also keeps the
  // written order: each fragment read and DMA issue sits between MFMAs.
  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      // the zeros are in place before the prologue below: the compiler does
      // not see the MFMAs inside the asm, so it would not space a register
      // write and the product that reads it apart
      asm volatile("" : "+a"(acc[i][j]));
    }
  auto mma = [&](int i, int j, const u32x4* fa, const u32x4* fb) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc[i][j]) : "v"(fa[i]), "v"(fb[j]));
  };
  u32x4 fa0[8], fb0[8], fa1[8], fb1[8];
#pragma unroll
  for (int q = 0; q < 16; ++q) dma1(0, 0, q);
  DR_WAIT_VM(0);
  DR_LDS_SYNC();
#pragma unroll
  for (int q = 0; q < 16; ++q) dma1(1, 1, q);
#pragma unroll
  for (int q = 0; q < 16; ++q) rd1(fa0, fb0, lds, 0, q);
  // Per 64-column step t (stage t & 1): the first half's products with the
  // second half's fragment reads between them; one barrier (step t + 1
  // landed everywhere, every wave done with stage t & 1); then the second
  // half's products with the DMA of step t + 2 into stage t & 1 and the reads
  // of step t + 1's first half between them.  Products accumulate in the
  // same order as a plain loop over 32-column halves.
  for (int t = 0; t < nk; ++t) {
    const unsigned char* sa = lds + (t & 1) * kBStage;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      rd1(fa1, fb1, sa, 1, q);
#pragma unroll
      for (int m = 4 * q; m < 4 * q + 4; ++m) mma(m & 7, m >> 3, fa0, fb0);
    }
    DR_WAIT_VM(0);
    DR_LDS_SYNC();
    const unsigned char* sn = lds + ((t + 1) & 1) * kBStage;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      dma1(t + 2, t & 1, q);
      rd1(fa0, fb0, sn, 0, q);
#pragma unroll
      for (int m = 4 * q; m < 4 * q + 4; ++m) mma(m & 7, m >> 3, fa1, fb1);
    }
  }
  // the last products' results are read below: wait states after an MFMA
  // that the compiler does not see inside the asm
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");

  float* Kp = a.K + (long long)p * a.n * a.n;
  if (a.vec4 && !diag && rowA0 + kBT <= a.n) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        big_store_block_fast(Kp, a.n, rowA0 + wr * 128 + 16 * i, rowB0 + wc * 128 + 16 * j, acc[i][j], lane);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        big_store_block_masked(Kp, a.n, diag, rowA0 + wr * 128 + 16 * i, rowB0 + wc * 128 + 16 * j, acc[i][j], lane);
  }
}

bool gram_use_big(int64_t n, int P, dr_dtype dtype) {
  if (dtype != DR_BF16 || n < 2 * kBT) return false;
  const int64_t T = (n + kBT - 1) / kBT;
  const int gp = P < kMaxGroups ? P : kMaxGroups;
  return T * (T + 1) / 2 * gp >= kBigMinTiles;
}

// One thread per element of a 64x64 tile: sums the chunk partials in chunk
// order and writes K (lower triangle and its mirror) and, for fp32 rows, s
// and t2 from the upper triangle of the diagonal tiles (where
// gram_tile_lds_kernel puts them).
__global__ __launch_bounds__(kThreads) void gram_reduce_kernel(GramArgs a, float* K, float* s, float* t2,
                                                               long long pbase) {
  const int q = blockIdx.x, p = blockIdx.y;
  const int e = blockIdx.z * kThreads + threadIdx.x;
  const long long width = a.goff[p + 1] - a.goff[p];
  const int nvalid = (int)((width + a.CK - 1) / a.CK);
  int I, J;
  pair_to_tiles(q, I, J);
  const int tr = e / kTile, tc = e % kTile;
  const int r = I * kTile + tr, c = J * kTile + tc;
  int srow = -1;   // >= 0: this element is s[srow]; -2: t2
  if (c <= r) {
    if (r >= a.n) return;
  } else if (a.rows > a.n && I == J) {
    if ((tr == 0 || tr == 16) && tc >= 32)
      srow = I * kTile + 2 * tr + (tc - 32);
    else if (I == 0 && tr == 0 && tc == 16)
      srow = -2;
    if (srow == -1 || srow >= a.n) return;
  } else {
    return;
  }
  const float* src = a.partial + ((long long)p * a.pairs + q) * a.maxchunks * (kTile * kTile) + e;
  // chunks in batches of 32 loads in flight, summed in chunk order
  float acc = 0.f;
  int ch = 0;
  for (; ch + 32 <= nvalid; ch += 32) {
    float v[32];
#pragma unroll
    for (int u = 0; u < 32; ++u) v[u] = src[(long long)(ch + u) * (kTile * kTile)];
#pragma unroll
    for (int u = 0; u < 32; ++u) acc += v[u];
  }
  for (; ch + 8 <= nvalid; ch += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[(long long)(ch + u) * (kTile * kTile)];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; ch < nvalid; ++ch) acc += src[(long long)ch * (kTile * kTile)];
  if (srow == -1) {
    float* Kp = K + (pbase + p) * (long long)a.n * a.n;
    Kp[(long long)r * a.n + c] = acc;
    Kp[(long long)c * a.n + r] = acc;
  } else if (srow >= 0) {
    s[(pbase + p) * (long long)a.n + srow] = acc;
  } else {
    t2[pbase + p] = acc;
  }
}

// gbar[c] = (1/m) sum_j Gt[j][c] for c in [c_lo, c_hi)
template <bool BF16>
__global__ __launch_bounds__(kThreads) void target_mean_kernel(const unsigned char* Gt, long long ldGt, int m,
                                                               long long c_lo, long long c_hi, float* gbar) {
  const long long c = c_lo + (long long)blockIdx.x * kThreads + threadIdx.x;
  if (c >= c_hi) return;
  auto ld = [&](int j) -> float {
    if constexpr (BF16) {
      const unsigned short h = reinterpret_cast<const unsigned short*>(Gt)[(long long)j * ldGt + c];
      return __uint_as_float((unsigned)h << 16);
    } else {
      return reinterpret_cast<const float*>(Gt)[(long long)j * ldGt + c];
    }
  };
  // rows in batches of 8 loads in flight, summed in row order
  double acc = 0.0;
  int j = 0;
  for (; j + 8 <= m; j += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = ld(j + u);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += (double)v[u];
  }
  for (; j < m; ++j) acc += (double)ld(j);
  gbar[c] = (float)(acc / (double)m);
}

// s[p][i] = <G[i][cols_p], gbar[cols_p]> for i < n; row n gives t2[p] = <gbar, gbar>.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void score_kernel(GramArgs a, const float* gbar, float* s, float* t2,
                                                         long long pbase) {
  const int i = blockIdx.x, p = blockIdx.y;
  const long long g0 = a.goff[p], g1 = a.goff[p + 1];
  double acc = 0.0;
  if (i < a.n) {
    // 16-byte loads: group edges are multiples of 8 (bf16) / 4 (fp32)
    // elements and rows are 16-byte aligned
    const unsigned char* row = a.G + (long long)i * a.ldG * GTr<BF16>::ES;
    constexpr int V = GTr<BF16>::EPV;
    for (long long c = g0 + (long long)threadIdx.x * V; c < g1; c += (long long)kThreads * V) {
      const u32x4 q = *reinterpret_cast<const u32x4*>(row + c * GTr<BF16>::ES);
      const float4 g4a = *reinterpret_cast<const float4*>(gbar + c);
      if constexpr (BF16) {
        const float4 g4b = *reinterpret_cast<const float4*>(gbar + c + 4);
        acc += (double)__uint_as_float(q.x << 16) * (double)g4a.x + (double)__uint_as_float(q.x & 0xffff0000u) * (double)g4a.y;
        acc += (double)__uint_as_float(q.y << 16) * (double)g4a.z + (double)__uint_as_float(q.y & 0xffff0000u) * (double)g4a.w;
        acc += (double)__uint_as_float(q.z << 16) * (double)g4b.x + (double)__uint_as_float(q.z & 0xffff0000u) * (double)g4b.y;
        acc += (double)__uint_as_float(q.w << 16) * (double)g4b.z + (double)__uint_as_float(q.w & 0xffff0000u) * (double)g4b.w;
      } else {
        acc += (double)__uint_as_float(q.x) * (double)g4a.x + (double)__uint_as_float(q.y) * (double)g4a.y;
        acc += (double)__uint_as_float(q.z) * (double)g4a.z + (double)__uint_as_float(q.w) * (double)g4a.w;
      }
    }
  } else {
    for (long long c = g0 + threadIdx.x; c < g1; c += kThreads) acc += (double)gbar[c] * (double)gbar[c];
  }
  __shared__ double red[kThreads];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (i < a.n)
      s[(pbase + p) * (long long)a.n + i] = (float)red[0];
    else
      t2[pbase + p] = (float)red[0];
  }
}

struct GramPlan {
  int64_t rows;
  int NT, pairs, CK, maxchunks;
  size_t gbar_bytes, partial_bytes;
  bool small;       // gram_small_kernel path
  int NRP;          // its padded row count
};

bool gram_use_small(int64_t n, dr_dtype dtype) { return dtype == DR_F32 && n >= 1 && n + 1 <= kSmMaxRows; }

// Chunk length: a multiple of 256 columns; for bf16 tiles shrunk until a
// launch has about kTargetWGs workgroups, for fp32 tiles sized to two
// rounds of kLdsSlots; identical for every launch of a call.
GramPlan gram_plan(int64_t n, const int64_t* goff, int P, dr_dtype dtype) {
  GramPlan g;
  // fp32 sketches: gbar joins as row n, so s and t2 come out of the same
  // pass (the tiles cover the n general rows; the diagonal tiles carry gbar)
  const int64_t rows = dtype == DR_F32 ? n + 1 : n;
  g.NT = (int)((n + kTile - 1) / kTile);
  g.pairs = g.NT * (g.NT + 1) / 2;
  int64_t maxw = 0;
  for (int p = 0; p < P; ++p) maxw = goff[p + 1] - goff[p] > maxw ? goff[p + 1] - goff[p] : maxw;
  const int gp = P < kMaxGroups ? P : kMaxGroups;
  int64_t ck = align_up((size_t)(maxw > 0 ? maxw : 1), 256);
  if (dtype == DR_F32) {
    // fp32 tiles: the chunk length that keeps the launch just within two
    // rounds of the workgroups the chip holds at once (kLdsSlots), so the
    // second round is nearly full (the fixed count keeps the chunking, and
    // with it the summation order, the same on every device)
    const int64_t want = ((int64_t)maxw * g.pairs * gp + 2 * kLdsSlots - 1) / (2 * kLdsSlots);
    const int64_t c2 = (int64_t)align_up((size_t)(want > 256 ? want : 256), 256);
    if (c2 < ck) ck = c2;
  } else {
    while (ck > 256 && (int64_t)g.pairs * gp * ((maxw + ck - 1) / ck) < kTargetWGs) ck = align_up((size_t)(ck / 2), 256);
  }
  g.CK = (int)ck;
  g.maxchunks = (int)((maxw + ck - 1) / ck);
  if (g.maxchunks < 1) g.maxchunks = 1;
  g.gbar_bytes = align_up((size_t)(goff[P] > 0 ? goff[P] : 1) * sizeof(float), 256);
  g.partial_bytes = (size_t)gp * g.pairs * g.maxchunks * kTile * kTile * sizeof(float);
  if (rows == 0 || gram_use_big(n, P, dtype)) g.partial_bytes = 0;
  g.rows = rows;
  g.small = gram_use_small(n, dtype);
  g.NRP = (int)((n + 1 + 15) / 16 * 16);
  if (g.small) {
    g.maxchunks = (int)((maxw + kSmCK - 1) / kSmCK);
    if (g.maxchunks < 1) g.maxchunks = 1;
    g.partial_bytes = (size_t)gp * g.maxchunks * g.NRP * g.NRP * sizeof(float);
  }
  return g;
}

dr_status gram_validate(const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt,
                        dr_dtype dtype, const int64_t* goff, int P, float* K, float* s, float* t2) {
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (!goff || P < 1 || n < 0 || m < 1 || n > (1 << 20)) return DR_ERR_ARG;
  if (goff[0] < 0) return DR_ERR_ARG;
  for (int p = 0; p < P; ++p)
    if (goff[p + 1] < goff[p]) return DR_ERR_ARG;
  const int64_t vec = dtype == DR_BF16 ? 8 : 4;
  if (ldGt < goff[P] || ldGt % vec || !Gt || !aligned16(Gt) || !t2) return DR_ERR_ARG;
  if (n > 0) {
    if (ldG < goff[P] || ldG % vec || !G || !aligned16(G) || !K || !s) return DR_ERR_ARG;
    for (int p = 0; p <= P; ++p)
      if (goff[p] % vec) return DR_ERR_ARG;
  }
  return DR_OK;
}

}  // namespace
}  // namespace dr

extern "C" size_t dr_gram_workspace_size(int64_t n, int64_t m, const int64_t* goff, int P, dr_dtype dtype) {
  (void)m;
  if (dtype != DR_BF16 && dtype != DR_F32) return 0;
  if (!goff || P < 1 || n < 0) return 0;
  dr::GramPlan g = dr::gram_plan(n, goff, P, dtype);
  return g.gbar_bytes + g.partial_bytes;
}

namespace dr {
namespace {

// host checks of a call (before any HIP call), then the plan
dr_status gram_check(const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt, dr_dtype dtype,
                     const int64_t* goff, int P, float* K, float* s, float* t2, GramPlan* plan) {
  dr_status st = gram_validate(G, n, ldG, Gt, m, ldGt, dtype, goff, P, K, s, t2);
  if (st != DR_OK) return st;
  // the large-n kernel addresses a 256-row panel with 32-bit buffer offsets
  if (gram_use_big(n, P, dtype) && (uint64_t)ldG * 2 * (kBT + 1) >= (uint64_t)kOobOffset) return DR_ERR_UNSUPPORTED;
  *plan = gram_plan(n, goff, P, dtype);
  return DR_OK;
}

// enqueue the Gram on hs with the workspace at `workspace` (every byte of
// it that a kernel reads is written earlier in the same call)
dr_status gram_run(const GramPlan& g, const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt,
                   dr_dtype dtype, const int64_t* goff, int P, float* K, float* s, float* t2, void* workspace,
                   hipStream_t hs) {
  dr_status st = DR_OK;
  const bool bf = dtype == DR_BF16;
  float* gbar = static_cast<float*>(workspace);
  float* partial = reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) + g.gbar_bytes);

  const long long c_lo = goff[0], c_hi = goff[P];
  if (c_hi > c_lo && !g.small) {   // the small path forms gbar inside its chunks
    const int blocks = (int)((c_hi - c_lo + kThreads - 1) / kThreads);
    if (bf)
      hipLaunchKernelGGL(target_mean_kernel<true>, dim3(blocks), dim3(kThreads), 0, hs,
                         static_cast<const unsigned char*>(Gt), (long long)ldGt, (int)m, c_lo, c_hi, gbar);
    else
      hipLaunchKernelGGL(target_mean_kernel<false>, dim3(blocks), dim3(kThreads), 0, hs,
                         static_cast<const unsigned char*>(Gt), (long long)ldGt, (int)m, c_lo, c_hi, gbar);
    if ((st = launch_status()) != DR_OK) return st;
  }

  for (int p0 = 0; p0 < P; p0 += kMaxGroups) {
    const int gp = P - p0 < kMaxGroups ? P - p0 : kMaxGroups;
    GramArgs a = {};
    a.G = static_cast<const unsigned char*>(G);
    a.ldG = ldG;
    a.n = (int)n;
    a.rows = (int)g.rows;
    a.gbar = gbar;
    for (int p = 0; p <= gp; ++p) a.goff[p] = goff[p0 + p];
    a.P = gp;
    a.NT = g.NT;
    a.pairs = g.pairs;
    a.CK = g.CK;
    a.maxchunks = g.maxchunks;
    a.partial = partial;
    a.K = K;
    a.s = s;
    a.t2 = t2;
    a.pbase = p0;
    if (gram_use_big(n, P, dtype)) {
      BigArgs b = {};
      b.G = static_cast<const unsigned char*>(G);
      b.ldG = ldG;
      b.n = (int)n;
      b.T = (int)((n + kBT - 1) / kBT);
      b.pairs = b.T * (b.T + 1) / 2;
      for (int p = 0; p <= gp; ++p) b.goff[p] = goff[p0 + p];
      b.K = K + (long long)p0 * n * n;
      int chunks = 0;
      for (int band = 0; 4 * band < b.T; ++band) chunks += ((4 * band + 4 < b.T ? 4 * band + 4 : b.T) + 7) / 8;
      b.vec4 = (n % 4 == 0) && aligned16(K);
      hipLaunchKernelGGL(gram_big_kernel, dim3((chunks + 7) / 8 * 256, gp), dim3(256), 0, hs, b);
      if ((st = launch_status()) != DR_OK) return st;
    } else if (g.small) {
      hipLaunchKernelGGL(gram_small_kernel, dim3(g.maxchunks, gp), dim3(kSmThreads), 0, hs, a,
                         static_cast<const float*>(Gt), (long long)ldGt, (int)m, g.NRP, g.maxchunks);
      if ((st = launch_status()) != DR_OK) return st;
      const int nr = (int)n + 1;
      hipLaunchKernelGGL(gram_small_reduce_kernel, dim3((nr * (nr + 1) / 2 + kThreads / 64 - 1) / (kThreads / 64), gp),
                         dim3(kThreads), 0, hs, a, g.NRP, g.maxchunks, K, s, t2, (long long)p0);
      if ((st = launch_status()) != DR_OK) return st;
    } else if (g.pairs > 0) {
      dim3 grid(g.maxchunks, g.pairs, gp);
      if (bf)
        hipLaunchKernelGGL(gram_tile_kernel<true>, grid, dim3(kThreads), 0, hs, a);
      else
        hipLaunchKernelGGL(gram_tile_lds_kernel, grid, dim3(kThreads), 0, hs, a);
      if ((st = launch_status()) != DR_OK) return st;
      if (bf || g.maxchunks > 1) {   // fp32 tiles of a single chunk are written by the tile kernel
        hipLaunchKernelGGL(gram_reduce_kernel, dim3(g.pairs, gp, kTile * kTile / kThreads), dim3(kThreads), 0, hs,
                           a, K, s, t2, (long long)p0);
        if ((st = launch_status()) != DR_OK) return st;
      }
    }
    if (bf) {
      // bf16 sketches: s and t2 against the fp32 target mean in a separate pass
      hipLaunchKernelGGL(score_kernel<true>, dim3(n + 1, gp), dim3(kThreads), 0, hs, a, gbar, s, t2, (long long)p0);
      if ((st = launch_status()) != DR_OK) return st;
    } else if (g.pairs == 0) {
      // fp32 with no general rows: t2 alone
      hipLaunchKernelGGL(score_kernel<false>, dim3(1, gp), dim3(kThreads), 0, hs, a, gbar, s, t2, (long long)p0);
      if ((st = launch_status()) != DR_OK) return st;
    }
  }
  return DR_OK;
}

}  // namespace
}  // namespace dr

extern "C" dr_status dr_gram(const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt,
                             dr_dtype dtype, const int64_t* goff, int P, float* K, float* s, float* t2,
                             void* workspace, size_t ws_bytes, void* stream) {
  dr::GramPlan g;
  const dr_status st = dr::gram_check(G, n, ldG, Gt, m, ldGt, dtype, goff, P, K, s, t2, &g);
  if (st != DR_OK) return st;
  if (!workspace || ws_bytes < g.gbar_bytes + g.partial_bytes) return DR_ERR_WORKSPACE;
  return dr::gram_run(g, G, n, ldG, Gt, m, ldGt, dtype, goff, P, K, s, t2, workspace,
                      reinterpret_cast<hipStream_t>(stream));
}

// ---------------------------------------------------------------------------
// dr_gram_noalloc: the same Gram with its workspace in a fixed device array.
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device (hipGetSymbolAddress, with
// that device current) and only that address is ever handed to a kernel.
// Each device holds its own copy of the array until the process ends.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[DR_GRAM_NOALLOC_MAX_BYTES];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices];   // device address of `scratch` per device, null until looked up
}  // namespace

extern "C" dr_status dr_gram_noalloc(const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt,
                                     dr_dtype dtype, const int64_t* goff, int P, float* K, float* s, float* t2,
                                     void* stream) {
  dr::GramPlan g;
  const dr_status st = dr::gram_check(G, n, ldG, Gt, m, ldGt, dtype, goff, P, K, s, t2, &g);
  if (st != DR_OK) return st;
  if (g.gbar_bytes + g.partial_bytes > (size_t)DR_GRAM_NOALLOC_MAX_BYTES) return DR_ERR_TOO_LARGE;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return DR_ERR_HIP;
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
      void* p = nullptr;
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DR_ERR_HIP;
      g_scratch_ptr[dev] = p;
    }
    ptr = g_scratch_ptr[dev];
  }
  return dr::gram_run(g, G, n, ldG, Gt, m, ldGt, dtype, goff, P, K, s, t2, ptr, reinterpret_cast<hipStream_t>(stream));
}
