// Factorised per-example gradient sketches of linear layers (dr_sketch_grads).
//
// For example i and layer l the sketch is P_out G_i P_in^T with
// G_i = sum_{t < len_i} dy_{i,t} x_{i,t}^T (per-sample weight gradient,
// Sec. 4.1; factorised compression of App. C.3 with the identity as
// second-stage projector).  G_i is never formed: per token tile
//   stage 1:  Y = X P_in^T  [tokens x k_in],  D = dY P_out^T  [tokens x k_out]
//             (bf16 or fp32 MFMA, fp32 accumulate, contraction over d)
//   stage 2:  S += D^T Y    [k_out x k_in]  (contraction over tokens)
// The stage-1 accumulators feed stage 2 straight from registers: the MFMA
// output layout (token 4*(l/16)+j, column l%16 in register j) is exactly the
// fp32-MFMA operand layout once token 4*(l/16)+j is read as the reduction
// index l/16 of the j-th product.  On the bf16 path stage 2 instead runs
// as three bf16 MFMAs on hi/lo bf16 splits of D and Y (Dh Yh + Dh Yl +
// Dl Yh), one MFMA per 32 rows.
//
// Two kernels do the work.  sketch_packed_kernel (below) is the main path:
// the valid tokens are packed into 128-token tiles and streamed HBM -> LDS
// by DMA through a three-stage ring; a workgroup walks a range of tiles
// (one tile, or an equal share of the layer's tokens when the launch is too
// small to fill the chip many times over).  sketch_kernel, the general
// fallback (d not a whole number of 64-element steps, or offsets beyond
// 32 bits), works on (layer, example, chunk of tokens) units: a 256-thread
// workgroup owns one unit and walks it in 128-token tiles, each of its four
// waves owning 32 tokens; x / dy rows stream from HBM straight into
// registers, the projector chunk shared by the four waves is staged in LDS
// (double buffered, one barrier per step), rows at or beyond the valid
// length are never loaded.  In both, the four per-wave partial sketches
// are summed through LDS in a fixed order and multi-part results are summed
// by a second kernel in a fixed order.  No atomics: results are
// deterministic, and padding may hold any bits.

#include "common.h"

namespace dr {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTokWave = 32;                  // tokens per wave per tile
constexpr int kTokTile = kWaves * kTokWave;   // tokens per workgroup tile
constexpr int kMaxLayersPerLaunch = 16;
constexpr int kTargetUnits = 2048;            // aim for >= 8 units per CU
constexpr int kXcds = 8;                      // accelerator dies; workgroups are dealt to them round robin

struct LayerArg {
  const unsigned char* x;
  const unsigned char* dy;
  const unsigned char* p_in;
  const unsigned char* p_out;
  long long ldx, lddy;   // elements
  int d_in, d_out;
  long long col_offset;
};

struct SketchArgs {
  LayerArg L[kMaxLayersPerLaunch];
  int num_layers;
  int N, T;
  int chunk_tokens;   // multiple of kTokTile
  int nchunks;
  const int* len;
  float* S;
  long long ldS;
  float* partial;     // [num_layers][N][nchunks][KOUT*KIN] when nchunks > 1
};

template <bool BF16>
struct Tr;
template <>
struct Tr<true> {
  static constexpr int ES = 2;     // bytes per element
  static constexpr int EPV = 8;    // elements per 16-byte vector
  static constexpr int KSUB = 32;  // reduction length covered by one 16-byte vector per lane
};
template <>
struct Tr<false> {
  static constexpr int ES = 4;
  static constexpr int EPV = 4;
  static constexpr int KSUB = 16;
};

// One 16-byte operand pair: for bf16 one 16x16x32 MFMA, for fp32 four
// 16x16x4 MFMAs (element h of lane group g is reduction index 4g+h).
template <bool BF16>
__device__ __forceinline__ f32x4 mma_vec(u32x4 a, u32x4 b, f32x4 c) {
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

__device__ __forceinline__ u32x4 ld16(const unsigned char* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

template <bool BF16, int KIN, int KOUT>
__global__ __launch_bounds__(kThreads, 2) void sketch_kernel(SketchArgs a) {
  using E = Tr<BF16>;
  constexpr int KC = 4 * E::KSUB;          // reduction elements per step
  constexpr int ROWB = KC * E::ES;         // 256 bytes of one projector row per step
  constexpr int RS = ROWB + 16;            // padded LDS row stride (conflict-free b128 reads)
  constexpr int KP = KIN > KOUT ? KIN : KOUT;
  constexpr int TI = KIN / 16, TO = KOUT / 16;
  constexpr int PVEC = KP * (ROWB / 16) / kThreads;   // projector vectors per thread per step
  constexpr int LDS_P = 2 * KP * RS;
  constexpr int LDS_R = kWaves * KOUT * KIN * 4;   // stage-2 partial sums, one region per wave
  constexpr int LDS_BYTES = LDS_P > LDS_R ? LDS_P : LDS_R;
  static_assert(PVEC >= 1 && PVEC * kThreads * 16 == KP * ROWB, "projector staging");
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = lane & 15;   // row within a 16-row MFMA block
  const int lg = lane >> 4;   // lane group (reduction slice)

  const int unit = blockIdx.x;
  const int chunk = unit % a.nchunks;
  const int ex = (unit / a.nchunks) % a.N;
  const int li = unit / (a.nchunks * a.N);
  const LayerArg& L = a.L[li];

  int len = a.T;
  if (a.len) {
    len = a.len[ex];
    len = len < 0 ? 0 : (len > a.T ? a.T : len);
  }
  const int t_begin = chunk * a.chunk_tokens;
  int t_end = t_begin + a.chunk_tokens;
  t_end = t_end < len ? t_end : len;

  f32x4 Sacc[TO][TI];
#pragma unroll
  for (int i = 0; i < TO; ++i)
#pragma unroll
    for (int j = 0; j < TI; ++j) Sacc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t_begin < t_end) {
    const int nsx = (L.d_in + KC - 1) / KC;
    const int nsd = (L.d_out + KC - 1) / KC;
    const int steps_per_tile = nsx + nsd;
    const int ntiles = (t_end - t_begin + kTokTile - 1) / kTokTile;
    const int nsteps = ntiles * steps_per_tile;

    // decode a global step index into (tile start, pass, k0)
    auto decode = [&](int s, int& t0, int& pass, int& k0) {
      const int tile = s / steps_per_tile;
      const int r = s - tile * steps_per_tile;
      t0 = t_begin + tile * kTokTile;
      pass = r < nsx ? 0 : 1;
      k0 = (pass == 0 ? r : r - nsx) * KC;
    };

    auto load_x = [&](int s, u32x4 (&xr)[2][4]) {
      int t0, pass, k0;
      decode(s, t0, pass, k0);
      const unsigned char* base = pass == 0 ? L.x : L.dy;
      const long long ld = pass == 0 ? L.ldx : L.lddy;
      const int d = pass == 0 ? L.d_in : L.d_out;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const int tok = t0 + wave * kTokWave + rb * 16 + lr;
        const bool tok_ok = tok < t_end;
        const unsigned char* row = base + ((long long)ex * a.T + tok) * ld * E::ES;
#pragma unroll
        for (int sub = 0; sub < 4; ++sub) {
          const int k = k0 + sub * E::KSUB + lg * E::EPV;
          if (tok_ok && k < d)
            xr[rb][sub] = ld16(row + (long long)k * E::ES);
          else
            xr[rb][sub] = u32x4{0u, 0u, 0u, 0u};
        }
      }
    };

    auto load_p = [&](int s, u32x4 (&pr)[PVEC]) {
      int t0, pass, k0;
      decode(s, t0, pass, k0);
      const unsigned char* P = pass == 0 ? L.p_in : L.p_out;
      const int rows = pass == 0 ? KIN : KOUT;
      const int d = pass == 0 ? L.d_in : L.d_out;
#pragma unroll
      for (int q = 0; q < PVEC; ++q) {
        const int v = tid + q * kThreads;
        const int row = v / (ROWB / 16);
        const int c16 = v % (ROWB / 16);
        const int k = k0 + c16 * E::EPV;
        if (row < rows && k < d)
          pr[q] = ld16(P + ((long long)row * d + k) * E::ES);
        else
          pr[q] = u32x4{0u, 0u, 0u, 0u};
      }
    };

    auto store_p = [&](int buf, const u32x4 (&pr)[PVEC]) {
#pragma unroll
      for (int q = 0; q < PVEC; ++q) {
        const int v = tid + q * kThreads;
        const int row = v / (ROWB / 16);
        const int c16 = v % (ROWB / 16);
        *reinterpret_cast<u32x4*>(lds + buf * KP * RS + row * RS + c16 * 16) = pr[q];
      }
    };

    f32x4 Y[2][TI], D[2][TO];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
      for (int c = 0; c < TI; ++c) Y[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < TO; ++c) D[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    u32x4 xr[2][4], xn[2][4], pn[PVEC];
    load_x(0, xr);
    load_p(0, pn);
    store_p(0, pn);
    __syncthreads();

    for (int s = 0; s < nsteps; ++s) {
      const bool more = s + 1 < nsteps;
      if (more) {
        load_x(s + 1, xn);
        load_p(s + 1, pn);
      }
      const int r = s % steps_per_tile;
      const int pass = r < nsx ? 0 : 1;
      const unsigned char* pb = lds + (s & 1) * KP * RS;
      if (pass == 0) {
#pragma unroll
        for (int sub = 0; sub < 4; ++sub) {
#pragma unroll
          for (int c = 0; c < TI; ++c) {
            const u32x4 b = *reinterpret_cast<const u32x4*>(pb + (c * 16 + lr) * RS + sub * 64 + lg * 16);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) Y[rb][c] = mma_vec<BF16>(xr[rb][sub], b, Y[rb][c]);
          }
        }
      } else {
#pragma unroll
        for (int sub = 0; sub < 4; ++sub) {
#pragma unroll
          for (int c = 0; c < TO; ++c) {
            const u32x4 b = *reinterpret_cast<const u32x4*>(pb + (c * 16 + lr) * RS + sub * 64 + lg * 16);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) D[rb][c] = mma_vec<BF16>(xr[rb][sub], b, D[rb][c]);
          }
        }
      }
      if (r == steps_per_tile - 1) {
        // stage 2: S += D^T Y over this tile's 32 tokens of this wave
#pragma unroll
        for (int o = 0; o < TO; ++o)
#pragma unroll
          for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
#pragma unroll
              for (int j = 0; j < 4; ++j) Sacc[o][i] = mma_f32(D[rb][o][j], Y[rb][i][j], Sacc[o][i]);
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
          for (int c = 0; c < TI; ++c) Y[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < TO; ++c) D[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
      if (more) store_p((s + 1) & 1, pn);
      __syncthreads();
      if (more) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int sub = 0; sub < 4; ++sub) xr[rb][sub] = xn[rb][sub];
      }
    }

    // sum the four waves' partial sketches in a fixed order:
    // (w0 + w2) + (w1 + w3)
    float* red = reinterpret_cast<float*>(lds);
    constexpr int SW = KOUT * KIN;   // floats per wave partial
    auto put = [&](int region) {
#pragma unroll
      for (int o = 0; o < TO; ++o)
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) red[region * SW + ((o * TI + i) * 4 + q) * 64 + lane] = Sacc[o][i][q];
    };
    auto add = [&](int region) {
#pragma unroll
      for (int o = 0; o < TO; ++o)
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) Sacc[o][i][q] += red[region * SW + ((o * TI + i) * 4 + q) * 64 + lane];
    };
    if (wave >= 2) put(wave - 2);
    __syncthreads();
    if (wave < 2) add(wave);
    __syncthreads();
    if (wave == 1) put(0);
    __syncthreads();
    if (wave == 0) add(0);
  }

  if (wave != 0) return;
  float* out;
  if (a.nchunks == 1) {
    out = a.S + (long long)ex * a.ldS + L.col_offset;
  } else {
    if (t_begin >= t_end) return;   // the reduction skips chunks past the valid length
    out = a.partial + ((long long)(li * a.N + ex) * a.nchunks + chunk) * (KOUT * KIN);
  }
#pragma unroll
  for (int o = 0; o < TO; ++o)
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) out[(o * 16 + lg * 4 + q) * KIN + i * 16 + lr] = Sacc[o][i][q];
}


// ---------------------------------------------------------------------------
// Packed-token streaming kernel (the main path).
//
// The valid tokens of every layer are taken in example order, as if the
// padded batch were packed: position p = cum[i] + t is token t < len_i of
// example i.  A workgroup owns one 128-token tile of packed positions of one
// layer, so every tile is full (up to the last one of the layer) whatever
// the length mix, and padding is never addressed.  A tile may hold the end
// of one example and the start of the next: stage 2 then runs once per
// example of the tile with the other examples' rows masked out of Y.  An
// example that lies inside one tile is written to S directly; an example
// spread over several tiles leaves one partial per tile (slot 0 if it is
// the tile's first example, else slot 1) that sketch_packed_reduce_kernel
// sums in tile order.
//
// Data movement: x / dy rows and projector chunks go HBM -> LDS with the
// buffer-to-LDS DMA (16 bytes per lane, no registers held while in flight)
// through a three-stage ring, so two steps of loads are outstanding while
// the current step computes.  Waits are explicit (vmcnt counts this wave's
// outstanding DMAs); the barrier is a bare s_barrier after lgkmcnt(0), so no
// fence drains the ring.
//
// LDS layout of a stage: every 16-row operand block (16 token rows of x or
// dy, or 16 projector rows) occupies 2 KiB as two halves of 8 rows x 128 B.
// One DMA instruction fills one half: lane l moves 16 bytes of row l/8, so
// each instruction reads eight whole 128-byte row segments from HBM.  The
// 16-byte slot of segment g of row r (r = 0..15 within the block) is
// g ^ (r % 8) ^ (r / 8); with that swizzle the MFMA operand reads
// (ds_read_b128, lane = row % 16 + 16 * reduction slice) hit all 64 banks
// exactly once per 16-lane phase.  x / dy DMAs are marked non-temporal: each
// element is read once.


// The packed positions [0, total) of a layer are split into WL ranges of
// R positions (R >= 128, computed on the device from total), one range per
// workgroup, each walked in up to KS tiles of 128 positions.  With WL =
// ceil(N T / 128) (R = 128, KS = 1) this is one tile per workgroup; for
// launches too small to fill the chip several times over, WL is chosen so
// that every workgroup of the launch is resident at once and each streams
// the same number of tokens, which removes the partly filled last round.
struct PackArgs {
  LayerArg L[kMaxLayersPerLaunch];
  int num_layers;
  int N, T;
  int WL, KS;           // workgroups per layer, tiles per workgroup (upper bound)
  int xcd;              // 1: number workgroups XCD by XCD (all layers of the launch alike)
  int out_vec4;         // 1: S rows and every layer's column offset are 16-byte aligned
  int max_tiles;        // WL * KS: tile slots per layer
  const int* cum;       // [N + 2]: exclusive prefix of the clamped lengths, then R
  const int* tile_ex;   // [max_tiles] example holding the first position of each tile, -1 if empty
  float* S;
  long long ldS;
  float* partial;       // [num_layers][max_tiles][2][KOUT * KIN]
};

// Exclusive prefix of the clamped lengths and the first example of each
// tile (one workgroup; N is small next to the streamed data).
__global__ __launch_bounds__(1024) void sketch_plan_kernel(const int* len, int N, int T, int WL, int KS, int* cum,
                                                           int* tile_ex) {
  __shared__ int wsum[17];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (N + 1023) / 1024;
  const int i0 = tid * per, i1 = i0 + per < N ? i0 + per : N;
  int loc = 0;
  for (int i = i0; i < i1; ++i) {
    int l = len ? len[i] : T;
    loc += l < 0 ? 0 : (l > T ? T : l);
  }
  int inc = loc;
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(inc, off, 64);
    if (lane >= off) inc += v;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < 16; ++w) {
      const int v = wsum[w];
      wsum[w] = run;
      run += v;
    }
    wsum[16] = run;
  }
  __syncthreads();
  int base = wsum[wave] + inc - loc;
  for (int i = i0; i < i1; ++i) {
    cum[i] = base;
    int l = len ? len[i] : T;
    base += l < 0 ? 0 : (l > T ? T : l);
  }
  const int total = wsum[16];
  const int share = (total + WL - 1) / WL;
  const int R = share > kTokTile ? share : kTokTile;   // positions per workgroup
  if (tid == 0) {
    cum[N] = total;
    cum[N + 1] = R;
  }
  __syncthreads();
  for (int tt = tid; tt < WL * KS; tt += 1024) {
    const int w = tt / KS, k = tt - w * KS;
    const int p = w * R + k * kTokTile;
    const int hi_w = w * R + R < total ? w * R + R : total;
    if (p >= hi_w) {
      tile_ex[tt] = -1;
      continue;
    }
    int lo = 0, hi = N;   // last e with cum[e] <= p
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cum[mid] <= p)
        lo = mid;
      else
        hi = mid - 1;
    }
    tile_ex[tt] = lo;
  }
}

// two fp32 values -> their bf16 truncations (hi, low half first) and the
// bf16 truncations of the remainders (lo)
__device__ __forceinline__ uint2 split_pack(float a, float b) {
  const unsigned ua = __float_as_uint(a), ub = __float_as_uint(b);
  const float ra = a - __uint_as_float(ua & 0xffff0000u);
  const float rb = b - __uint_as_float(ub & 0xffff0000u);
  return make_uint2((ua >> 16) | (ub & 0xffff0000u), (__float_as_uint(ra) >> 16) | (__float_as_uint(rb) & 0xffff0000u));
}

template <bool BF16, int KIN, int KOUT>
__global__ __launch_bounds__(kThreads, 2) void sketch_packed_kernel(PackArgs a) {
  using E = Tr<BF16>;
  constexpr int NSUB = 2;                   // MFMA operand vectors per row per step
  constexpr int KC = NSUB * E::KSUB;        // 64 bf16 / 32 fp32 elements per step
  constexpr int KP = KIN > KOUT ? KIN : KOUT;
  constexpr int TI = KIN / 16, TO = KOUT / 16, TPM = KP / 16;
  constexpr int XBLK = kWaves * 2 * NSUB;   // 16 x blocks of 1 KiB
  constexpr int PBLK = 2 * TPM > 4 ? 2 * TPM : 4;
  constexpr int NPW = PBLK / kWaves;        // projector DMAs per wave per stage
  constexpr int NDMA = 2 * NSUB + NPW;      // DMAs per wave per stage
  constexpr int STAGE = (XBLK + PBLK) * 1024;
  constexpr int NST = 3;
  constexpr int LDS_R = kWaves * KOUT * KIN * 4;   // stage-2 partial sums, one region per wave
  // the ring (or the stage-2 partial sums), then the tile's prefix entries
  constexpr int LDS_MAIN = NST * STAGE > LDS_R ? NST * STAGE : LDS_R;
  constexpr int LDS_BYTES = LDS_MAIN + 1024;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[LDS_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4, hr = lane >> 3;
  // XCD-aware numbering (layers of one shape): workgroups are dealt to the
  // 8 XCDs round robin, so the (layer, range) index v gives each XCD a
  // contiguous run of ranges and a layer's projector chunks stay in few
  // XCDs' L2 (one when the launch holds a multiple of 8 layers).  With layers
  // of different sizes the runs would leave some XCDs idle, so the plain
  // order is kept.
  const int G8 = a.xcd ? (int)gridDim.x / kXcds : 0;
  const int b = blockIdx.x;
  const int v = b < G8 * kXcds ? (b % kXcds) * G8 + b / kXcds : b;
  const int li = v / a.WL;
  const int wg = v - li * a.WL;
  const int total = a.cum[a.N];
  const int R = a.cum[a.N + 1];
  const int r_lo = wg * R;
  const int r_hi = r_lo + R < total ? r_lo + R : total;
  const LayerArg& L = a.L[li];
  const int* cum = a.cum;
  for (int kt = 0; kt < a.KS; ++kt) {
  const int p0 = r_lo + kt * kTokTile;
  const int pend = p0 + kTokTile < r_hi ? p0 + kTokTile : r_hi;   // this tile's positions: [p0, pend)
  if (p0 >= pend) break;
  const int tile = wg * a.KS + kt;
  const int e0 = a.tile_ex[tile];
  // cum[e0 .. e0 + 128] staged once in LDS.  A tile holds at most 128
  // non-empty examples; runs of empty ones in between can only push an
  // example past the staged range, which then reads cum from memory.
  int* tcum = reinterpret_cast<int*>(lds + LDS_MAIN);   // kTokTile + 1 entries
  __syncthreads();   // the previous tile is done with tcum and the ring
  {
    const int r = tid;
    if (r <= kTokTile && e0 + r <= a.N) tcum[r] = cum[e0 + r];
  }
  __syncthreads();
  auto cumat = [&](int r) { return r <= kTokTile ? tcum[r] : cum[e0 + r]; };

  // example (relative to e0) and token of a packed position, -1 past the tile
  auto locate = [&](int p, int& rel, int& tok) {
    if (p >= pend) {
      rel = -1;
      tok = 0;
      return;
    }
    int r = 0;
    while (cumat(r + 1) <= p) ++r;
    rel = r;
    tok = p - cumat(r);
  };
  // byte offsets of this lane's DMA rows (rb, half) from the tile's base example
  unsigned offx[2][2], offd[2][2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      int rel, tok;
      locate(p0 + wave * kTokWave + rb * 16 + h * 8 + hr, rel, tok);
      const long long row = (long long)rel * a.T + tok;
      offx[rb][h] = rel < 0 ? kOobOffset : (unsigned)(row * L.ldx * E::ES);
      offd[rb][h] = rel < 0 ? kOobOffset : (unsigned)(row * L.lddy * E::ES);
    }
  int e_last;
  {
    int rel, tok;
    locate(pend - 1, rel, tok);
    e_last = e0 + rel;
  }

  const __amdgpu_buffer_rsrc_t rx = make_rsrc(L.x + (long long)e0 * a.T * L.ldx * E::ES, kOobOffset);
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(L.dy + (long long)e0 * a.T * L.lddy * E::ES, kOobOffset);
  const __amdgpu_buffer_rsrc_t rpi = make_rsrc(L.p_in, (unsigned)(KIN * L.d_in * E::ES));
  const __amdgpu_buffer_rsrc_t rpo = make_rsrc(L.p_out, (unsigned)(KOUT * L.d_out * E::ES));
  const int nsx = L.d_in / KC, nsd = L.d_out / KC;
  const int nsteps = nsx + nsd;
  const unsigned seg0 = (unsigned)swz_seg_of_lane(lane, 0), seg1 = (unsigned)swz_seg_of_lane(lane, 1);

  // issue every DMA of step s into ring stage st
  auto issue = [&](int s, int st) {
    const int pass = s < nsx ? 0 : 1;
    const unsigned k0 = (unsigned)((pass == 0 ? s : s - nsx) * KC);
    unsigned char* sb = lds + st * STAGE;
    const __amdgpu_buffer_rsrc_t rr = pass == 0 ? rx : rd;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const unsigned ro = pass == 0 ? offx[rb][h] : offd[rb][h];
        const unsigned off = ro == kOobOffset ? kOobOffset : ro + (k0 + (h ? seg1 : seg0) * E::EPV) * E::ES;
        dma16<kAuxStream>(rr, sb + ((wave * 2 + rb) * 2 + h) * 1024, off);
      }
    const __amdgpu_buffer_rsrc_t rp = pass == 0 ? rpi : rpo;
    const unsigned dp = (unsigned)(pass == 0 ? L.d_in : L.d_out);
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
      const int b = wave + j * kWaves;          // projector half block (column tile, half)
      const int ct = b >> 1, h = b & 1;
      const unsigned row = (unsigned)(ct * 16 + h * 8 + hr);
      // blocks past the projector's tiles and rows past k_in / k_out fall
      // outside the descriptor's range and fill with zeros
      const unsigned off = ct < TPM ? (row * dp + k0 + (h ? seg1 : seg0) * E::EPV) * E::ES : kOobOffset;
      dma16<0>(rp, sb + (XBLK + b) * 1024, off);
    }
  };

  f32x4 Y[2][TI], D[2][TO];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
    for (int c = 0; c < TI; ++c) Y[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < TO; ++c) D[rb][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  issue(0, 0);
  if (nsteps > 1) issue(1, 1);
  int st = 0;
  // steps [s0, s1) of one pass accumulate into ACC (Y for x, D for dy); the
  // two passes are separate loops so each accumulates in place
  auto pass_steps = [&](int s0, int s1, auto& ACC) {
    constexpr int NC = sizeof(ACC[0]) / sizeof(f32x4);
    for (int s = s0; s < s1; ++s) {
      if (s + 1 < nsteps)
        DR_WAIT_VM(NDMA);
      else
        DR_WAIT_VM(0);
      DR_LDS_SYNC();
      if (s + 2 < nsteps) issue(s + 2, st == 0 ? 2 : st - 1);
      const unsigned char* sb = lds + st * STAGE;
      // operand (row lr, reduction slice lg of sub-step sub) = segment sub*4 + lg
      u32x4 xf[2][NSUB];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int sub = 0; sub < NSUB; ++sub) xf[rb][sub] = swz_read(sb + (wave * 2 + rb) * 2048, lr, sub * 4 + lg);
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const u32x4 b = swz_read(sb + (XBLK + 2 * c) * 1024, lr, sub * 4 + lg);
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) ACC[rb][c] = mma_vec<BF16>(xf[rb][sub], b, ACC[rb][c]);
        }
      st = st == 2 ? 0 : st + 1;
    }
  };
  pass_steps(0, nsx, Y);
  pass_steps(nsx, nsteps, D);
  DR_LDS_SYNC();

  // stage 2 once per example of the tile, the other examples' rows masked.
  // Each wave writes its partial sums to its own LDS region one 16-row
  // block of the output at a time (few live registers), then all threads
  // add the four regions in the fixed order (w0 + w2) + (w1 + w3).
  float* red = reinterpret_cast<float*>(lds);
  constexpr int SW = KOUT * KIN;
  // packed position of the first row this lane holds in the MFMA outputs
  // (rows rbase + rb*16 + j, j < 4)
  const int rbase = p0 + wave * kTokWave + lg * 4;
  const int wlo = p0 + wave * kTokWave, whi = wlo + kTokWave;   // this wave's rows
  // bf16 sketches: each fp32 stage-1 output v is split as hi + lo with hi =
  // v truncated to bf16 and lo = (v - hi) truncated to bf16, and
  // sum_t D Y ~ Dh Yh + Dh Yl + Dl Yh (relative error about 3 * 2^-16 per
  // product).  One 16x16x32 bf16 MFMA then covers the wave's 32 rows: lane
  // group g holds rows {4g + j, 16 + 4g + j}, which become the 8 consecutive
  // reduction indices of its operand, for D and Y alike.
  u32x4 Dh[TO], Dl[TO];
  if constexpr (BF16) {
#pragma unroll
    for (int o = 0; o < TO; ++o) {
      { const uint2 s_ = split_pack(D[0][o][0], D[0][o][1]); Dh[o].x = s_.x; Dl[o].x = s_.y; }
      { const uint2 s_ = split_pack(D[0][o][2], D[0][o][3]); Dh[o].y = s_.x; Dl[o].y = s_.y; }
      { const uint2 s_ = split_pack(D[1][o][0], D[1][o][1]); Dh[o].z = s_.x; Dl[o].z = s_.y; }
      { const uint2 s_ = split_pack(D[1][o][2], D[1][o][3]); Dh[o].w = s_.x; Dl[o].w = s_.y; }
    }
  }
  for (int e = e0; e <= e_last; ++e) {
    const int ce = cumat(e - e0), ce1 = cumat(e - e0 + 1);
    if (ce1 == ce) continue;   // empty examples are written by the reduction kernel
    const bool all_e = ce <= wlo && ce1 >= whi;   // every row of the wave belongs to e
    const bool some_e = ce < whi && ce1 > wlo;
    if constexpr (BF16) {
      u32x4 Yh[TI], Yl[TI];
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        float y[2][4];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int pr = rbase + rb * 16 + j;
            y[rb][j] = (all_e || (pr >= ce && pr < ce1)) ? Y[rb][i][j] : 0.f;
          }
        { const uint2 s_ = split_pack(y[0][0], y[0][1]); Yh[i].x = s_.x; Yl[i].x = s_.y; }
        { const uint2 s_ = split_pack(y[0][2], y[0][3]); Yh[i].y = s_.x; Yl[i].y = s_.y; }
        { const uint2 s_ = split_pack(y[1][0], y[1][1]); Yh[i].z = s_.x; Yl[i].z = s_.y; }
        { const uint2 s_ = split_pack(y[1][2], y[1][3]); Yh[i].w = s_.x; Yl[i].w = s_.y; }
      }
#pragma unroll
      for (int o = 0; o < TO; ++o)
#pragma unroll
        for (int i = 0; i < TI; ++i) {
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
          if (some_e) {
            acc = mma_bf16(Dh[o], Yh[i], acc);
            acc = mma_bf16(Dh[o], Yl[i], acc);
            acc = mma_bf16(Dl[o], Yh[i], acc);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) red[wave * SW + ((o * TI + i) * 4 + q) * 64 + lane] = acc[q];
        }
    } else {
#pragma unroll
    for (int o = 0; o < TO; ++o) {
      f32x4 Sacc[TI];
#pragma unroll
      for (int i = 0; i < TI; ++i) Sacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (all_e) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int j = 0; j < 4; ++j) Sacc[i] = mma_f32(D[rb][o][j], Y[rb][i][j], Sacc[i]);
      } else if (some_e) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int pr = rbase + rb * 16 + j;
              Sacc[i] = mma_f32(D[rb][o][j], (pr >= ce && pr < ce1) ? Y[rb][i][j] : 0.f, Sacc[i]);
            }
      }
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) red[wave * SW + ((o * TI + i) * 4 + q) * 64 + lane] = Sacc[i][q];
    }
    }
    DR_LDS_SYNC();
    const bool inside = ce >= p0 && ce1 <= pend;
    float* out = inside ? a.S + (long long)e * a.ldS + L.col_offset
                        : a.partial + (((long long)li * a.max_tiles + tile) * 2 + (e == e0 ? 0 : 1)) * SW;
    if (!inside || a.out_vec4) {
      // four consecutive lanes' entries are four consecutive columns of one
      // output row: float4 reads of the four regions and one float4 store
      for (int k = 4 * tid; k < SW; k += 4 * kThreads) {
        const float4 r0 = *reinterpret_cast<const float4*>(&red[k]);
        const float4 r1 = *reinterpret_cast<const float4*>(&red[SW + k]);
        const float4 r2 = *reinterpret_cast<const float4*>(&red[2 * SW + k]);
        const float4 r3 = *reinterpret_cast<const float4*>(&red[3 * SW + k]);
        const float4 v = make_float4((r0.x + r2.x) + (r1.x + r3.x), (r0.y + r2.y) + (r1.y + r3.y),
                                     (r0.z + r2.z) + (r1.z + r3.z), (r0.w + r2.w) + (r1.w + r3.w));
        const int l = k & 63, oiq = k >> 6;           // (o * TI + i) * 4 + q
        const int q = oiq & 3, oi = oiq >> 2;
        const int o = oi / TI, i = oi - o * TI;
        *reinterpret_cast<float4*>(&out[(o * 16 + (l >> 4) * 4 + q) * KIN + i * 16 + (l & 15)]) = v;
      }
    } else {
      for (int k = tid; k < SW; k += kThreads) {
        const float v = (red[k] + red[2 * SW + k]) + (red[SW + k] + red[3 * SW + k]);
        const int l = k & 63, oiq = k >> 6;           // (o * TI + i) * 4 + q
        const int q = oiq & 3, oi = oiq >> 2;
        const int o = oi / TI, i = oi - o * TI;
        out[(o * 16 + (l >> 4) * 4 + q) * KIN + i * 16 + (l & 15)] = v;
      }
    }
    DR_LDS_SYNC();
  }
  }   // tiles of this workgroup
}

// Examples spread over several tiles: sum their per-tile partials in tile
// order (eight tiles' loads in flight); empty examples get zeros.  One float4
// of the sketch block per thread, kPackReduceWGs workgroups per (layer,
// example).
template <int KIN, int KOUT>
constexpr int kPackReduceWGs = (KOUT * KIN / 4 + kThreads - 1) / kThreads;

template <int KIN, int KOUT>
__global__ __launch_bounds__(kThreads) void sketch_packed_reduce_kernel(PackArgs a) {
  constexpr int V4 = KOUT * KIN / 4;
  constexpr int NP = kPackReduceWGs<KIN, KOUT>;
  const int part = blockIdx.x % NP;
  const int pair = blockIdx.x / NP;
  const int li = pair / a.N, e = pair % a.N;
  const int ce = a.cum[e], ce1 = a.cum[e + 1];
  const int R = a.cum[a.N + 1];
  // tile slot of a position: workgroup p / R, tile (p mod R) / 128 within it
  const int t0 = (ce / R) * a.KS + (ce % R) / kTokTile;
  const int t1 = ((ce1 - 1) / R) * a.KS + ((ce1 - 1) % R) / kTokTile;
  if (ce1 > ce && t0 == t1) return;   // written by its only tile
  const int e4 = part * kThreads + threadIdx.x;
  if (e4 >= V4) return;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  if (ce1 > ce) {
    // partial of tile tt, slot sl: [layer][tile][slot][KOUT * KIN]
    const f32x4* base = reinterpret_cast<const f32x4*>(a.partial + (long long)li * a.max_tiles * 2 * (KOUT * KIN)) + e4;
    for (int tb = t0; tb <= t1; tb += 8) {
      int ex[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) ex[u] = tb + u <= t1 ? a.tile_ex[tb + u] : -1;   // < 0: no partial
      f32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[u] = ex[u] >= 0 ? base[(long long)((tb + u) * 2 + (ex[u] == e ? 0 : 1)) * V4] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (ex[u] >= 0) acc += v[u];
    }
  }
  float* out = a.S + (long long)e * a.ldS + a.L[li].col_offset;
  out[4 * e4 + 0] = acc[0];
  out[4 * e4 + 1] = acc[1];
  out[4 * e4 + 2] = acc[2];
  out[4 * e4 + 3] = acc[3];
}

constexpr int kReduceSplit = 4;   // workgroups per (layer, example) of sketch_reduce_kernel

// Sum the chunk partials of every (layer, example) in chunk order (register
// kernel path): four workgroups per (layer, example), one float4 per thread.
template <int KIN, int KOUT>
__global__ __launch_bounds__(kThreads) void sketch_reduce_kernel(SketchArgs a) {
  constexpr int V4 = KOUT * KIN / 4;
  constexpr int PER = (V4 + kReduceSplit * kThreads - 1) / (kReduceSplit * kThreads);
  const int part = blockIdx.x % kReduceSplit;
  const int pair = blockIdx.x / kReduceSplit;
  const int li = pair / a.N, ex = pair % a.N;
  int len = a.T;
  if (a.len) {
    len = a.len[ex];
    len = len < 0 ? 0 : (len > a.T ? a.T : len);
  }
  const int nvalid = (len + a.chunk_tokens - 1) / a.chunk_tokens;
  const f32x4* p = reinterpret_cast<const f32x4*>(a.partial + (long long)(li * a.N + ex) * a.nchunks * (KOUT * KIN));
  float* out = a.S + (long long)ex * a.ldS + a.L[li].col_offset;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e4 = (part * PER + u) * kThreads + threadIdx.x;
    if (e4 >= V4) break;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    int c = 0;
    for (; c + 4 <= nvalid; c += 4) {
      f32x4 v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = p[(long long)(c + q) * V4 + e4];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc += v[q];
    }
    for (; c < nvalid; ++c) acc += p[(long long)c * V4 + e4];
    out[4 * e4 + 0] = acc[0];
    out[4 * e4 + 1] = acc[1];
    out[4 * e4 + 2] = acc[2];
    out[4 * e4 + 3] = acc[3];
  }
}

// ---------------------------------------------------------------------------
// Host side: planning and dispatch.

bool valid_k(int64_t k) { return k == 16 || k == 32 || k == 64; }

// Layers are grouped into launches of at most kMaxLayersPerLaunch
// consecutive layers with equal (k_in, k_out).  A launch takes the packed
// path when d_in and d_out are whole numbers of steps and every byte offset
// a tile can form (at most min(N, 128) examples from its first one) fits in
// 32 bits; otherwise the register kernel runs over (layer, example, chunk)
// units whose chunk length is halved (in whole tiles) until the launch has
// at least kTargetUnits units.
struct Launch {
  int first, count, kin, kout, chunk, nchunks;
  bool packed;
};

struct Plan {
  int nlaunch;
  int WL, KS, max_tiles;
  size_t off_cum, off_tiles, off_partial, bytes;
};

// resident packed workgroups per CU (LDS-bound) times the CU count
int resident_slots() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus < 1)
    cus = 256;
  return 2 * cus;
}

int64_t packed_tiles(int64_t N, int64_t T) { return (N * T + kTokTile - 1) / kTokTile; }

bool packed_ok(const dr_layer* layers, int first, int count, int64_t N, int64_t T, dr_dtype dtype) {
  const int64_t kc = dtype == DR_BF16 ? 64 : 32;
  const int64_t es = dtype == DR_BF16 ? 2 : 4;
  const int64_t span = (N < kTokTile ? N : kTokTile) * T + kTokTile;
  for (int j = first; j < first + count; ++j) {
    const dr_layer& L = layers[j];
    if (L.d_in % kc || L.d_out % kc) return false;
    const int64_t ld = L.ldx > L.lddy ? L.ldx : L.lddy;
    if ((uint64_t)span * (uint64_t)ld * (uint64_t)es >= (uint64_t)kOobOffset) return false;
  }
  return true;
}

Plan plan(const dr_layer* layers, int num_layers, int64_t N, int64_t T, dr_dtype dtype, Launch* out) {
  Plan pl = {};
  size_t need = 0;
  bool any_packed = false;
  const int64_t mt = packed_tiles(N, T);
  // balanced ranges when the largest packed launch has at most 8 tiles per
  // resident workgroup slot (else one tile per workgroup)
  int lmax = 0;
  for (int i0 = 0; i0 < num_layers;) {
    int j0 = i0 + 1;
    while (j0 < num_layers && j0 - i0 < kMaxLayersPerLaunch && layers[j0].k_in == layers[i0].k_in &&
           layers[j0].k_out == layers[i0].k_out)
      ++j0;
    if (packed_ok(layers, i0, j0 - i0, N, T, dtype) && j0 - i0 > lmax) lmax = j0 - i0;
    i0 = j0;
  }
  int64_t WL = mt, KS = 1;
  if (lmax > 0 && mt > 0) {
    const int64_t slots = resident_slots();
    if ((int64_t)lmax * mt <= 8 * slots) {
      WL = slots / lmax;
      if (WL < 1) WL = 1;
      if (WL > mt) WL = mt;
      const int64_t share = (N * T + WL - 1) / WL;   // upper bound of R
      KS = (share + kTokTile - 1) / kTokTile;
    }
  }
  pl.WL = (int)WL;
  pl.KS = (int)KS;
  const int64_t slots_per_layer = WL * KS;
  int i = 0;
  while (i < num_layers) {
    int j = i + 1;
    while (j < num_layers && j - i < kMaxLayersPerLaunch && layers[j].k_in == layers[i].k_in &&
           layers[j].k_out == layers[i].k_out)
      ++j;
    Launch l = {};
    l.first = i;
    l.count = j - i;
    l.kin = (int)layers[i].k_in;
    l.kout = (int)layers[i].k_out;
    l.packed = packed_ok(layers, i, l.count, N, T, dtype);
    if (l.packed) {
      any_packed = true;
      l.chunk = kTokTile;
      l.nchunks = 1;
      const size_t b = (size_t)l.count * slots_per_layer * 2 * l.kin * l.kout * sizeof(float);
      if (b > need) need = b;
    } else {
      int64_t tiles = (T + kTokTile - 1) / kTokTile;
      if (tiles < 1) tiles = 1;
      int64_t chunk_tiles = tiles;
      while (chunk_tiles > 1 && (int64_t)l.count * N * ((tiles + chunk_tiles - 1) / chunk_tiles) < kTargetUnits)
        chunk_tiles = (chunk_tiles + 1) / 2;
      l.chunk = (int)(chunk_tiles * kTokTile);
      l.nchunks = (int)((tiles + chunk_tiles - 1) / chunk_tiles);
      if (l.nchunks > 1) {
        const size_t b = (size_t)l.count * N * l.nchunks * l.kin * l.kout * sizeof(float);
        if (b > need) need = b;
      }
    }
    if (out) out[pl.nlaunch] = l;
    ++pl.nlaunch;
    i = j;
  }
  pl.max_tiles = (int)slots_per_layer;
  if (any_packed) {
    pl.off_cum = 0;
    pl.off_tiles = align_up((size_t)(N + 2) * sizeof(int), 256);
    pl.off_partial = pl.off_tiles + align_up((size_t)(slots_per_layer > 0 ? slots_per_layer : 1) * sizeof(int), 256);
  } else {
    pl.off_cum = pl.off_tiles = pl.off_partial = 0;
  }
  pl.bytes = (need > 0 || any_packed) && N > 0 ? pl.off_partial + need : 0;
  return pl;
}

template <bool BF16, int KIN, int KOUT>
void launch_t(const Launch& l, const SketchArgs& a, const PackArgs& pa, hipStream_t st) {
  if (l.packed) {
    if (pa.max_tiles > 0)
      hipLaunchKernelGGL((sketch_packed_kernel<BF16, KIN, KOUT>), dim3(l.count * pa.WL), dim3(kThreads), 0, st, pa);
    hipLaunchKernelGGL((sketch_packed_reduce_kernel<KIN, KOUT>), dim3(l.count * pa.N * kPackReduceWGs<KIN, KOUT>), dim3(kThreads),
                       0, st, pa);
    return;
  }
  const int units = l.count * a.N * l.nchunks;
  hipLaunchKernelGGL((sketch_kernel<BF16, KIN, KOUT>), dim3(units), dim3(kThreads), 0, st, a);
  if (a.nchunks > 1)
    hipLaunchKernelGGL((sketch_reduce_kernel<KIN, KOUT>), dim3(a.num_layers * a.N * kReduceSplit), dim3(kThreads), 0,
                       st, a);
}

template <bool BF16>
void launch_k(const Launch& l, const SketchArgs& a, const PackArgs& pa, hipStream_t st) {
#define DR_SK(I, O)                               \
  if (l.kin == I && l.kout == O) {                \
    launch_t<BF16, I, O>(l, a, pa, st);           \
    return;                                       \
  }
  DR_SK(16, 16) DR_SK(16, 32) DR_SK(16, 64)
  DR_SK(32, 16) DR_SK(32, 32) DR_SK(32, 64)
  DR_SK(64, 16) DR_SK(64, 32) DR_SK(64, 64)
#undef DR_SK
}

dr_status validate(const dr_layer* layers, int num_layers, int64_t N, int64_t T, dr_dtype dtype,
                   const float* S, int64_t ldS) {
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (!layers || num_layers < 1 || N < 0 || T < 0) return DR_ERR_ARG;
  if (N > (1 << 24) || T > (1 << 24) || N * T > (1LL << 31) - kTokTile) return DR_ERR_ARG;
  const int64_t vec = dtype == DR_BF16 ? 8 : 4;
  if (N > 0 && !S) return DR_ERR_ARG;
  for (int l = 0; l < num_layers; ++l) {
    const dr_layer& L = layers[l];
    if (!valid_k(L.k_in) || !valid_k(L.k_out)) return DR_ERR_ARG;
    if (L.d_in < 1 || L.d_out < 1 || L.d_in % vec || L.d_out % vec) return DR_ERR_ARG;
    if (L.d_in > (1 << 28) || L.d_out > (1 << 28)) return DR_ERR_ARG;
    if (L.ldx < L.d_in || L.lddy < L.d_out || L.ldx % vec || L.lddy % vec) return DR_ERR_ARG;
    if (L.col_offset < 0 || L.col_offset + L.k_in * L.k_out > ldS) return DR_ERR_ARG;
    if (!L.p_in || !L.p_out || !aligned16(L.p_in) || !aligned16(L.p_out)) return DR_ERR_ARG;
    if (N > 0 && T > 0) {
      if (!L.x || !L.dy || !aligned16(L.x) || !aligned16(L.dy)) return DR_ERR_ARG;
    }
  }
  return DR_OK;
}

}  // namespace
}  // namespace dr

extern "C" size_t dr_sketch_workspace_size(const dr_layer* layers, int num_layers, int64_t N, int64_t T,
                                           dr_dtype dtype) {
  if (!layers || num_layers < 1 || N < 0 || T < 0) return 0;
  if (dtype != DR_BF16 && dtype != DR_F32) return 0;
  for (int l = 0; l < num_layers; ++l)
    if (!dr::valid_k(layers[l].k_in) || !dr::valid_k(layers[l].k_out)) return 0;
  return dr::plan(layers, num_layers, N, T, dtype, nullptr).bytes;
}

extern "C" dr_status dr_sketch_grads(const dr_layer* layers, int num_layers, int64_t N, int64_t T,
                                     const int32_t* len, dr_dtype dtype, float* S, int64_t ldS,
                                     void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  dr_status st = validate(layers, num_layers, N, T, dtype, S, ldS);
  if (st != DR_OK) return st;
  const Plan pl = plan(layers, num_layers, N, T, dtype, nullptr);
  if (pl.bytes > 0 && (!workspace || ws_bytes < pl.bytes)) return DR_ERR_WORKSPACE;
  if (N == 0) return DR_OK;
  Launch* lv = new Launch[pl.nlaunch];
  plan(layers, num_layers, N, T, dtype, lv);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  bool planned = false;
  for (int q = 0; q < pl.nlaunch && st == DR_OK; ++q) {
    const Launch& l = lv[q];
    SketchArgs a = {};
    PackArgs pa = {};
    // layers with the most bytes per token first: the launch's last
    // workgroups then stream the smallest tiles, which shortens its tail
    // (outputs go to each layer's own column range, so the order is free)
    int ord[kMaxLayersPerLaunch];
    for (int j = 0; j < l.count; ++j) {
      int p = j;
      const int64_t wj = layers[l.first + j].d_in + layers[l.first + j].d_out;
      while (p > 0 && layers[l.first + ord[p - 1]].d_in + layers[l.first + ord[p - 1]].d_out < wj) {
        ord[p] = ord[p - 1];
        --p;
      }
      ord[p] = j;
    }
    for (int j = 0; j < l.count; ++j) {
      const dr_layer& L = layers[l.first + ord[j]];
      LayerArg la;
      la.x = static_cast<const unsigned char*>(L.x);
      la.dy = static_cast<const unsigned char*>(L.dy);
      la.p_in = static_cast<const unsigned char*>(L.p_in);
      la.p_out = static_cast<const unsigned char*>(L.p_out);
      la.ldx = L.ldx;
      la.lddy = L.lddy;
      la.d_in = (int)L.d_in;
      la.d_out = (int)L.d_out;
      la.col_offset = L.col_offset;
      a.L[j] = la;
      pa.L[j] = la;
    }
    a.num_layers = pa.num_layers = l.count;
    pa.xcd = 1;
    for (int j = 1; j < l.count; ++j)
      if (pa.L[j].d_in != pa.L[0].d_in || pa.L[j].d_out != pa.L[0].d_out) pa.xcd = 0;
    pa.out_vec4 = aligned16(S) && ldS % 4 == 0;
    for (int j = 0; j < l.count; ++j)
      if (pa.L[j].col_offset % 4 != 0) pa.out_vec4 = 0;
    a.N = pa.N = (int)N;
    a.T = pa.T = (int)T;
    a.chunk_tokens = l.chunk;
    a.nchunks = l.nchunks;
    a.len = len;
    a.S = pa.S = S;
    a.ldS = pa.ldS = ldS;
    a.partial = reinterpret_cast<float*>(ws);
    if (l.packed) {
      pa.WL = pl.WL;
      pa.KS = pl.KS;
      pa.max_tiles = pl.max_tiles;
      pa.cum = reinterpret_cast<const int*>(ws + pl.off_cum);
      pa.tile_ex = reinterpret_cast<const int*>(ws + pl.off_tiles);
      pa.partial = reinterpret_cast<float*>(ws + pl.off_partial);
      if (!planned) {
        hipLaunchKernelGGL(sketch_plan_kernel, dim3(1), dim3(1024), 0, hs, len, (int)N, (int)T, pl.WL, pl.KS,
                           reinterpret_cast<int*>(ws + pl.off_cum), reinterpret_cast<int*>(ws + pl.off_tiles));
        if ((st = launch_status()) != DR_OK) break;
        planned = true;
      }
    }
    if (dtype == DR_BF16)
      launch_k<true>(l, a, pa, hs);
    else
      launch_k<false>(l, a, pa, hs);
    st = launch_status();
  }
  delete[] lv;
  return st;
}
