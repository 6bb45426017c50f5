// Factorised per-example gradient sketches of linear layers (dr_sketch_grads).
//
// For example i and layer l the sketch is P_out G_i P_in^T with
// G_i = sum_{t < len_i} dy_{i,t} x_{i,t}^T (per-sample weight gradient,
// Sec. 4.1; factorised compression of App. C.1 with the identity as
// second-stage projector).  G_i is never formed: per token tile
//   stage 1:  Y = X P_in^T  [tokens x k_in],  D = dY P_out^T  [tokens x k_out]
//             (bf16 or fp32 MFMA, fp32 accumulate, contraction over d)
//   stage 2:  S += D^T Y    [k_out x k_in]  (fp32 MFMA, contraction over tokens)
// The stage-1 accumulators feed stage 2 straight from registers: the MFMA
// output layout (token 4*(l/16)+j, column l%16 in register j) is exactly the
// fp32-MFMA operand layout once token 4*(l/16)+j is read as the reduction
// index l/16 of the j-th product.
//
// Work decomposition: a work unit is (layer, example, chunk of tokens); a
// 256-thread workgroup owns one unit and walks it in 128-token tiles, each
// of its four waves owning 32 tokens of the tile.  The x / dy rows stream
// from HBM straight into registers (each element is used by one wave only);
// the projector chunk shared by the four waves is staged once per step in
// LDS (double buffered, one barrier per step).  Rows at or beyond the valid
// length are never loaded (zero-filled), so padding may hold any bits.
// The four per-wave partial sketches are summed through LDS in a fixed
// order; with more than one chunk per example a second kernel sums the
// chunk partials in chunk order.  No atomics: results are deterministic.

#include "common.h"

namespace dr {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTokWave = 32;                  // tokens per wave per tile
constexpr int kTokTile = kWaves * kTokWave;   // tokens per workgroup tile
constexpr int kMaxLayersPerLaunch = 16;
constexpr int kTargetUnits = 2048;            // aim for >= 8 units per CU

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
  constexpr int LDS_R = 2 * KOUT * KIN * 4;
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

// Sum the chunk partials of every (layer, example) in chunk order.
template <int KIN, int KOUT>
__global__ __launch_bounds__(kThreads) void sketch_reduce_kernel(SketchArgs a) {
  const int li = blockIdx.x / a.N;
  const int ex = blockIdx.x % a.N;
  int len = a.T;
  if (a.len) {
    len = a.len[ex];
    len = len < 0 ? 0 : (len > a.T ? a.T : len);
  }
  const int nvalid = (len + a.chunk_tokens - 1) / a.chunk_tokens;
  const float* p = a.partial + (long long)(li * a.N + ex) * a.nchunks * (KOUT * KIN);
  float* out = a.S + (long long)ex * a.ldS + a.L[li].col_offset;
  for (int e = threadIdx.x; e < KOUT * KIN; e += kThreads) {
    float acc = 0.f;
    for (int c = 0; c < nvalid; ++c) acc += p[(long long)c * (KOUT * KIN) + e];
    out[e] = acc;
  }
}

template <bool BF16, int KIN, int KOUT>
void launch_t(const SketchArgs& a, int units, hipStream_t st) {
  hipLaunchKernelGGL((sketch_kernel<BF16, KIN, KOUT>), dim3(units), dim3(kThreads), 0, st, a);
  if (a.nchunks > 1)
    hipLaunchKernelGGL((sketch_reduce_kernel<KIN, KOUT>), dim3(a.num_layers * a.N), dim3(kThreads), 0, st, a);
}

template <bool BF16>
void launch_k(const SketchArgs& a, int units, int kin, int kout, hipStream_t st) {
#define DR_SK(I, O)                                        \
  if (kin == I && kout == O) {                             \
    launch_t<BF16, I, O>(a, units, st);                    \
    return;                                                \
  }
  DR_SK(16, 16) DR_SK(16, 32) DR_SK(16, 64)
  DR_SK(32, 16) DR_SK(32, 32) DR_SK(32, 64)
  DR_SK(64, 16) DR_SK(64, 32) DR_SK(64, 64)
#undef DR_SK
}

bool valid_k(int64_t k) { return k == 16 || k == 32 || k == 64; }

// Launch plan: layers are grouped into launches of at most
// kMaxLayersPerLaunch consecutive layers with equal (k_in, k_out); the chunk
// length is halved (in whole tiles) until a launch has >= kTargetUnits units.
struct Launch {
  int first, count, kin, kout, chunk, nchunks;
};

int plan(const dr_layer* layers, int num_layers, int64_t N, int64_t T, Launch* out, size_t* ws) {
  int nl = 0;
  size_t need = 0;
  int i = 0;
  while (i < num_layers) {
    int j = i + 1;
    while (j < num_layers && j - i < kMaxLayersPerLaunch && layers[j].k_in == layers[i].k_in &&
           layers[j].k_out == layers[i].k_out)
      ++j;
    Launch l;
    l.first = i;
    l.count = j - i;
    l.kin = (int)layers[i].k_in;
    l.kout = (int)layers[i].k_out;
    int64_t tiles = (T + kTokTile - 1) / kTokTile;
    if (tiles < 1) tiles = 1;
    int64_t chunk_tiles = tiles;
    while (chunk_tiles > 1 && (int64_t)l.count * N * ((tiles + chunk_tiles - 1) / chunk_tiles) < kTargetUnits)
      chunk_tiles = (chunk_tiles + 1) / 2;
    l.chunk = (int)(chunk_tiles * kTokTile);
    l.nchunks = (int)((tiles + chunk_tiles - 1) / chunk_tiles);
    if (l.nchunks > 1) {
      size_t b = (size_t)l.count * N * l.nchunks * l.kin * l.kout * sizeof(float);
      if (b > need) need = b;
    }
    if (out) out[nl] = l;
    ++nl;
    i = j;
  }
  if (ws) *ws = need;
  return nl;
}

dr_status validate(const dr_layer* layers, int num_layers, int64_t N, int64_t T, dr_dtype dtype,
                   const float* S, int64_t ldS) {
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (!layers || num_layers < 1 || N < 0 || T < 0) return DR_ERR_ARG;
  if (N > (1 << 24) || T > (1 << 24)) return DR_ERR_ARG;
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
  (void)dtype;
  if (!layers || num_layers < 1 || N < 0 || T < 0) return 0;
  for (int l = 0; l < num_layers; ++l)
    if (!dr::valid_k(layers[l].k_in) || !dr::valid_k(layers[l].k_out)) return 0;
  size_t ws = 0;
  dr::plan(layers, num_layers, N, T, nullptr, &ws);
  return ws;
}

extern "C" dr_status dr_sketch_grads(const dr_layer* layers, int num_layers, int64_t N, int64_t T,
                                     const int32_t* len, dr_dtype dtype, float* S, int64_t ldS,
                                     void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  dr_status st = validate(layers, num_layers, N, T, dtype, S, ldS);
  if (st != DR_OK) return st;
  size_t need = 0;
  const int nlaunch = plan(layers, num_layers, N, T, nullptr, &need);
  if (need > 0 && (!workspace || ws_bytes < need)) return DR_ERR_WORKSPACE;
  if (N == 0) return DR_OK;
  Launch* plan_buf = new Launch[nlaunch];
  plan(layers, num_layers, N, T, plan_buf, nullptr);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  for (int q = 0; q < nlaunch; ++q) {
    const Launch& l = plan_buf[q];
    SketchArgs a = {};
    for (int j = 0; j < l.count; ++j) {
      const dr_layer& L = layers[l.first + j];
      a.L[j].x = static_cast<const unsigned char*>(L.x);
      a.L[j].dy = static_cast<const unsigned char*>(L.dy);
      a.L[j].p_in = static_cast<const unsigned char*>(L.p_in);
      a.L[j].p_out = static_cast<const unsigned char*>(L.p_out);
      a.L[j].ldx = L.ldx;
      a.L[j].lddy = L.lddy;
      a.L[j].d_in = (int)L.d_in;
      a.L[j].d_out = (int)L.d_out;
      a.L[j].col_offset = L.col_offset;
    }
    a.num_layers = l.count;
    a.N = (int)N;
    a.T = (int)T;
    a.chunk_tokens = l.chunk;
    a.nchunks = l.nchunks;
    a.len = len;
    a.S = S;
    a.ldS = ldS;
    a.partial = static_cast<float*>(workspace);
    const int units = l.count * (int)N * l.nchunks;
    if (dtype == DR_BF16)
      launch_k<true>(a, units, l.kin, l.kout, hs);
    else
      launch_k<false>(a, units, l.kin, l.kout, hs);
    st = launch_status();
    if (st != DR_OK) break;
  }
  delete[] plan_buf;
  return st;
}
