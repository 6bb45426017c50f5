// Assembly of the update in full parameter space (dr_assemble_update):
//   U_l = sum_{i < n, w_i != 0} w_i sum_{t < len_i} dy_{i,t} x_{i,t}^T      (d_out x d_in)
// the post-hoc step of Sec. 4.2 that turns the weights of the retained
// examples into the layer updates (top-k weights 1/k on S give the subset
// mean g_S; span or cone weights give u = G^T w of Eq. (proj)).
//
// Kernels
//   update_plan_kernel   one workgroup per example list (one list per
//                        distinct weight row): the examples with w != 0 and
//                        len > 0, their clamped lengths and weights.
//   update_sort_kernel   orders each list by |w| ascending (index breaks
//                        ties) by ranking every entry against all others.
//   update_bf16_kernel   one 256 x 256 tile of U per workgroup, 8 waves of
//                        128 (d_out) x 64 (d_in).  Tokens go through a
//                        2-stage LDS ring in steps of 64 (64 KB a stage:
//                        the next step loads during the 64 MFMAs of this
//                        one, fewer and longer steps than 4 x 32), filled by
//                        buffer->LDS DMA in their natural token-major
//                        layout; both MFMA operands need 8 consecutive
//                        tokens per lane, which the gfx950 transposing LDS
//                        read (ds_read_b64_tr_b16) delivers straight from
//                        that layout.  One fp32 accumulator holds
//                        sum_e (w_e / w_cur) P_e: when the weight changes
//                        from w_cur to w_next it is multiplied by
//                        w_cur / w_next, and by the last weight at the end.
//                        The |w|-ascending order keeps every factor within
//                        [-1, 1] (no overflow whatever the weights), and a
//                        run of equal weights (all of them for top-k)
//                        costs no rescaling at all.
//   update_f32_kernel    fp32 inputs: 64 x 64 tiles, 4 waves of 32 x 32,
//                        fp32 MFMA 16x16x4, staged by plain loads; per
//                        example sums added to a second accumulator.
//   update_reduce_kernel when there are fewer tiles than CUs the example
//                        list of a tile is split over `split` workgroups;
//                        their partial tiles are summed in split order.
// Determinism: every sum runs in a fixed order (the sorted list, tokens
// ascending, splits ascending); no atomics.

#include "common.h"

namespace dr {
namespace {

constexpr int kMaxUpdLayers = 16;
constexpr int kMaxSplit = 32;

// bf16 tile
constexpr int kBO = 256, kBI = 256, kBK = 64;
constexpr int kBThreads = 512;
constexpr int kBDyBytes = kBK * kBO * 2;   // kBK token rows of 512 bytes
constexpr int kBXBytes = kBK * kBI * 2;
constexpr int kBNH = kBK / 16;             // 1 KB DMA blocks per operand per wave and step
constexpr int kBKK = kBK / 32;             // MFMA reduction slices per step
constexpr int kBStage = kBDyBytes + kBXBytes;
constexpr int kBStages = 2;

// f32 tile
constexpr int kFO = 64, kFI = 64, kFK = 16;
constexpr int kFThreads = 256;
constexpr int kFLd = 80;                   // LDS row stride (floats): the 4 rows of a b32 fragment read hit distinct banks

struct UpdLayerArg {
  const unsigned char* x;
  const unsigned char* dy;
  long long ldx, lddy;   // elements per token
  long long exx, exdy;   // bytes per example (T * ld * element size)
  int d_in, d_out;
  int ti;                // tiles along d_in
  int tile0;             // first tile of this layer within the launch
  int list;              // example list of this layer
  float* U;              // [d_out][d_in]
  const float* gstar;    // score mode: the target-mean gradient [d_out][d_in]
  double* part;          // score mode: partial scores [tiles of the layer][n]
};

struct UpdArgs {
  UpdLayerArg L[kMaxUpdLayers];
  int num_layers;
  int ntiles;            // tiles of the launch (all layers)
  int split;             // workgroups per tile along the example list
  int n;                 // list stride (>= 1)
  int nw;                // weighted examples (may be 0)
  const int* ex;         // [lists][n] selected examples, |w| ascending
  const int* exlen;      // [lists][n] their clamped lengths (> 0)
  const float* exw;      // [lists][n] their weights (!= 0)
  const int* cnt;        // [lists] list lengths
  int* uex;              // [lists][n] the same lists before sorting
  int* ulen;
  float* uw;
  float* partial;        // [ntiles * split][tile elements] when split > 1
};

// ------------------------------------------------------------------ plan

struct RowSel {
  int r[kMaxUpdLayers];   // weight row (group) of each layer slot
};

__global__ __launch_bounds__(1024) void update_plan_kernel(const float* w, long long ldw, UpdArgs a,
                                                           const int* len, int T, int list0, RowSel rs) {
  __shared__ int wsum[16];
  __shared__ int base_s;
  const int j = blockIdx.x;                 // layer slot of the launch
  const int list = list0 + j;
  const float* wr = w + (long long)rs.r[j] * ldw;
  int* ex = a.uex + (long long)list * a.n;
  int* exlen = a.ulen + (long long)list * a.n;
  float* exw = a.uw + (long long)list * a.n;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) base_s = 0;
  __syncthreads();
  for (int b = 0; b < a.nw; b += 1024) {
    const int i = b + tid;
    int L = 0;
    float wi = 0.f;
    if (i < a.nw) {
      wi = wr[i];
      L = len ? len[i] : T;
      L = L < 0 ? 0 : (L > T ? T : L);
    }
    const bool keep = i < a.nw && wi != 0.f && L > 0;
    const unsigned long long m = __ballot(keep);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    int off = base_s;
    for (int v = 0; v < wave; ++v) off += wsum[v];
    if (keep) {
      ex[off + before] = i;
      exlen[off + before] = L;
      exw[off + before] = wi;
    }
    __syncthreads();
    if (tid == 0) {
      int t = 0;
      for (int v = 0; v < 16; ++v) t += wsum[v];
      base_s += t;
    }
    __syncthreads();
  }
  if (tid == 0) const_cast<int*>(a.cnt)[list] = base_s;
}

// entry i of a list goes to position #{j : (|w_j|, ex_j) < (|w_i|, ex_i)}
__global__ __launch_bounds__(256) void update_sort_kernel(UpdArgs a) {
  __shared__ float kw[256];
  __shared__ int ki[256];
  const int list = blockIdx.y;
  const int cnt = a.cnt[list];
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x * 256 >= cnt) return;
  const long long base = (long long)list * a.n;
  const float wi = i < cnt ? fabsf(a.uw[base + i]) : 0.f;
  const int xi = i < cnt ? a.uex[base + i] : 0;
  int rank = 0;
  for (int j0 = 0; j0 < cnt; j0 += 256) {
    __syncthreads();
    const int j = j0 + threadIdx.x;
    kw[threadIdx.x] = j < cnt ? fabsf(a.uw[base + j]) : 0.f;
    ki[threadIdx.x] = j < cnt ? a.uex[base + j] : 0;
    __syncthreads();
    const int m = cnt - j0 < 256 ? cnt - j0 : 256;
    for (int q = 0; q < m; ++q) rank += (kw[q] < wi || (kw[q] == wi && ki[q] < xi)) ? 1 : 0;
  }
  if (i < cnt) {
    const_cast<int*>(a.ex)[base + rank] = xi;
    const_cast<int*>(a.exlen)[base + rank] = a.ulen[base + i];
    const_cast<float*>(a.exw)[base + rank] = a.uw[base + i];
  }
}

// which layer / tile / split a workgroup runs.  Workgroup b runs on XCD
// b % 8; each XCD takes a contiguous run of (tile, split) items, so the
// workgroups sharing an L2 share d_out panels of one layer.
__device__ __forceinline__ bool locate(const UpdArgs& a, int& layer, int& to, int& ti, int& s, int& item) {
  const int items = a.ntiles * a.split;
  const int per = (items + 7) >> 3;
  const int k = blockIdx.x >> 3;
  if (k >= per) return false;
  item = (blockIdx.x & 7) * per + k;
  if (item >= items) return false;
  const int tile = item / a.split;
  s = item - tile * a.split;
  layer = 0;
  while (layer + 1 < a.num_layers && a.L[layer + 1].tile0 <= tile) ++layer;
  const int t = tile - a.L[layer].tile0;
  to = t / a.L[layer].ti;
  ti = t - to * a.L[layer].ti;
  return true;
}

// ------------------------------------------------------------------ bf16


// SCORE = false: the update.  SCORE = true (the Direct scorer of Sec. 4.3):
// every example of the list gets weight 1; at the end of each example its
// tile of G_i is dotted with the same tile of the target-mean gradient and
// the accumulator cleared, so G_i is formed tile by tile and never stored.
template <bool SCORE>
__global__ __launch_bounds__(kBThreads) void update_bf16_kernel(UpdArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kBStages * kBStage];
  int layer, to, ti, s, item;
  if (!locate(a, layer, to, ti, s, item)) return;
  const UpdLayerArg& Lr = a.L[layer];
  const int d_in = Lr.d_in, d_out = Lr.d_out;
  const int o0 = to * kBO, i0 = ti * kBI;
  const int cnt = a.cnt[Lr.list];
  const int e_lo = (int)((long long)s * cnt / a.split), e_hi = (int)((long long)(s + 1) * cnt / a.split);
  const int* ex = a.ex + (long long)Lr.list * a.n;
  const int* exlen = a.exlen + (long long)Lr.list * a.n;
  const float* exw = a.exw + (long long)Lr.list * a.n;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // DMA roles: both tiles have kBK token rows of 512 bytes; wave w fills
  // rows 2j, 2j + 1 for j = w, w + 8, ... of each (1 KB per wave load).
  // Lane l fills 16 bytes: physical slot u / 2, half u % 2 of its row.
  int rrow[kBNH];
  unsigned cdy[kBNH], cx[kBNH];   // byte column inside a token row, or kOobOffset
#pragma unroll
  for (int h = 0; h < kBNH; ++h) {
    const int j = w + 8 * h;
    const int r = 2 * j + (lane >> 5), u = lane & 31;
    const int col = 16 * ((u >> 1) ^ slot_xor(r)) + 8 * (u & 1);
    rrow[h] = r;
    cdy[h] = o0 + col < d_out ? (unsigned)((o0 + col) * 2) : kOobOffset;
    cx[h] = i0 + col < d_in ? (unsigned)((i0 + col) * 2) : kOobOffset;
  }
  const unsigned rowb_dy = (unsigned)(Lr.lddy * 2), rowb_x = (unsigned)(Lr.ldx * 2);

  int ie = e_lo, it = 0, ilen = ie < e_hi ? exlen[ie] : 0;
  auto issue = [&](int st) {
    unsigned char* sb = lds + st * kBStage;
    __amdgpu_buffer_rsrc_t rdys, rxs;
    unsigned o_dy[kBNH], o_x[kBNH];
    if (ie < e_hi) {
      const long long e = ex[ie];
      rdys = make_rsrc(Lr.dy + e * Lr.exdy, kOobOffset);
      rxs = make_rsrc(Lr.x + e * Lr.exx, kOobOffset);
#pragma unroll
      for (int h = 0; h < kBNH; ++h) {
        const int t = it + rrow[h];
        o_dy[h] = (t < ilen && cdy[h] != kOobOffset) ? (unsigned)t * rowb_dy + cdy[h] : kOobOffset;
        o_x[h] = (t < ilen && cx[h] != kOobOffset) ? (unsigned)t * rowb_x + cx[h] : kOobOffset;
      }
      it += kBK;
      if (it >= ilen) {
        ++ie;
        it = 0;
        ilen = ie < e_hi ? exlen[ie] : 0;
      }
    } else {
      rdys = make_rsrc(Lr.dy, kOobOffset);
      rxs = make_rsrc(Lr.x, kOobOffset);
#pragma unroll
      for (int h = 0; h < kBNH; ++h) o_dy[h] = o_x[h] = kOobOffset;
    }
#pragma unroll
    for (int h = 0; h < kBNH; ++h) dma16<kAuxCached>(rdys, sb + (w + 8 * h) * 1024, o_dy[h]);
#pragma unroll
    for (int h = 0; h < kBNH; ++h) dma16<kAuxCached>(rxs, sb + kBDyBytes + (w + 8 * h) * 1024, o_x[h]);
  };

  // fragment reads: lane (g, q, r) of the transposing read addresses token
  // row 8g + q (+4 for the second half) and 8-byte piece r of the 16-column
  // block; the block's logical slot is XOR-ed with the row's swizzle.
  const int g = lane >> 4, q = (lane >> 2) & 3, rr = lane & 3;
  const int fx = q | ((g & 1) << 2);
  const int wr = w >> 2, wc = w & 3;   // 128-row half (d_out), 64-column quarter (d_in)
  const unsigned rbase = (unsigned)((8 * g + q) * 512 + rr * 8);
  unsigned offa[8], offb[4];
#pragma unroll
  for (int b = 0; b < 8; ++b) offa[b] = rbase + (unsigned)(((8 * wr + b) ^ fx) * 32);
#pragma unroll
  for (int b = 0; b < 4; ++b) offb[b] = kBDyBytes + rbase + (unsigned)(((4 * wc + b) ^ fx) * 32);

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  float wlast = 0.f;
  int ce = e_lo, ct = 0, clen = ce < e_hi ? exlen[ce] : 0;
  if (ce < e_hi) {
#pragma unroll
    for (int st = 0; st < kBStages - 1; ++st) issue(st);
    for (int step = 0; ce < e_hi; ++step) {
      DR_WAIT_VM(2 * kBNH * (kBStages - 2));   // this step's loads are done; later steps' may be in flight
      DR_LDS_SYNC();
      issue((step + kBStages - 1) % kBStages);
      const unsigned char* sb0 = lds + (step % kBStages) * kBStage;
#pragma unroll
      for (int kk = 0; kk < kBKK; ++kk) {
        const unsigned char* sb = sb0 + kk * 32 * 512;   // token rows 32 kk .. 32 kk + 31
        u32x4 fa[8], fb[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const v4s lo = lds_read_tr16(sb + offb[b]);
          const v4s hi = lds_read_tr16(sb + offb[b] + 4 * 512);
          fb[b] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                        __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
        }
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const v4s lo = lds_read_tr16(sb + offa[b]);
          const v4s hi = lds_read_tr16(sb + offa[b] + 4 * 512);
          fa[b] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                        __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mma_bf16(fa[i], fb[j], acc[i][j]);
      }
      ct += kBK;
      if (ct >= clen) {
        if constexpr (SCORE) {
          __shared__ double red[kBThreads / 64];
          const int lc = lane & 15;
          float d = 0.f;
#pragma unroll
          for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int o = o0 + 128 * wr + 16 * i + 4 * g + r;
              if (o >= d_out) continue;
              const float* grow = Lr.gstar + (long long)o * d_in;
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const int c = i0 + 64 * wc + 16 * j + lc;
                if (c < d_in) d = fmaf(acc[i][j][r], grow[c], d);
              }
            }
          double dd = (double)d;
          for (int off = 32; off > 0; off >>= 1) dd += __shfl_xor(dd, off, 64);
          if (lane == 0) red[w] = dd;
          __syncthreads();
          if (tid == 0) {
            double t = 0.0;
            for (int v = 0; v < kBThreads / 64; ++v) t += red[v];
            Lr.part[(long long)(to * Lr.ti + ti) * a.nw + ex[ce]] = t;
          }
          __syncthreads();
#pragma unroll
          for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
          ++ce;
          ct = 0;
          clen = ce < e_hi ? exlen[ce] : 0;
        } else {
          const float we = exw[ce];
          ++ce;
          ct = 0;
          clen = ce < e_hi ? exlen[ce] : 0;
          wlast = we;
          if (ce < e_hi) {
            const float wn = exw[ce];
            if (wn != we) {
              const float f = we / wn;   // |f| <= 1 in the sorted order
#pragma unroll
              for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                  for (int r = 0; r < 4; ++r) acc[i][j][r] *= f;
            }
          }
        }
      }
    }
    DR_WAIT_VM(0);
  }
  if constexpr (SCORE) return;

  // C layout: register r of block (i, j) is row 4g + r, column lane % 16
  const int lc = lane & 15;
  if (a.split == 1) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = o0 + 128 * wr + 16 * i + 4 * g + r;
        if (o >= d_out) continue;
        float* urow = Lr.U + (long long)o * d_in;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = i0 + 64 * wc + 16 * j + lc;
          if (c < d_in) urow[c] = wlast * acc[i][j][r];
        }
      }
  } else {
    float* P = a.partial + (long long)item * (kBO * kBI);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          P[(128 * wr + 16 * i + 4 * g + r) * kBI + 64 * wc + 16 * j + lc] = wlast * acc[i][j][r];
  }
}

// ------------------------------------------------------------------ f32

__global__ __launch_bounds__(kFThreads) void update_f32_kernel(UpdArgs a) {
  __shared__ __attribute__((aligned(16))) float sdy[2][kFK][kFLd];
  __shared__ __attribute__((aligned(16))) float sx[2][kFK][kFLd];
  int layer, to, ti, s, item;
  if (!locate(a, layer, to, ti, s, item)) return;
  const UpdLayerArg& Lr = a.L[layer];
  const int d_in = Lr.d_in, d_out = Lr.d_out;
  const int o0 = to * kFO, i0 = ti * kFI;
  const int cnt = a.cnt[Lr.list];
  const int e_lo = (int)((long long)s * cnt / a.split), e_hi = (int)((long long)(s + 1) * cnt / a.split);
  const int* ex = a.ex + (long long)Lr.list * a.n;
  const int* exlen = a.exlen + (long long)Lr.list * a.n;
  const float* exw = a.exw + (long long)Lr.list * a.n;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // staging: thread t loads token row t / 16 (of 16), columns 4 (t % 16) .. +3 of both operands
  const int sr = tid >> 4, sc = 4 * (tid & 15);
  const bool okdy = o0 + sc < d_out, okx = i0 + sc < d_in;
  float4 vdy = make_float4(0.f, 0.f, 0.f, 0.f), vx = vdy;
  int ie = e_lo, it = 0, ilen = ie < e_hi ? exlen[ie] : 0;
  auto fetch = [&]() {
    vdy = make_float4(0.f, 0.f, 0.f, 0.f);
    vx = vdy;
    if (ie < e_hi) {
      const long long e = ex[ie];
      const int t = it + sr;
      if (t < ilen) {
        if (okdy)
          vdy = *reinterpret_cast<const float4*>(Lr.dy + e * Lr.exdy + ((long long)t * Lr.lddy + o0 + sc) * 4);
        if (okx) vx = *reinterpret_cast<const float4*>(Lr.x + e * Lr.exx + ((long long)t * Lr.ldx + i0 + sc) * 4);
      }
      it += kFK;
      if (it >= ilen) {
        ++ie;
        it = 0;
        ilen = ie < e_hi ? exlen[ie] : 0;
      }
    }
  };

  const int wo = w >> 1, wi = w & 1;   // 32 x 32 quarter of the tile
  const int lr = lane & 15, lk = lane >> 4;
  f32x4 acc[2][2], tot[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      tot[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  int ce = e_lo, ct = 0, clen = ce < e_hi ? exlen[ce] : 0;
  if (ce < e_hi) fetch();
  for (int step = 0; ce < e_hi; ++step) {
    const int b = step & 1;
    *reinterpret_cast<float4*>(&sdy[b][sr][sc]) = vdy;
    *reinterpret_cast<float4*>(&sx[b][sr][sc]) = vx;
    __syncthreads();
    fetch();   // next step's loads in flight during this step's products
#pragma unroll
    for (int kk = 0; kk < kFK / 4; ++kk) {
      const int k = 4 * kk + lk;
      float fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = sdy[b][k][32 * wo + 16 * i + lr];
#pragma unroll
      for (int j = 0; j < 2; ++j) fb[j] = sx[b][k][32 * wi + 16 * j + lr];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mma_f32(fa[i], fb[j], acc[i][j]);
    }
    ct += kFK;
    if (ct >= clen) {
      const float we = exw[ce];
      ++ce;
      ct = 0;
      clen = ce < e_hi ? exlen[ce] : 0;
      if (ce >= e_hi || exw[ce] != we) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
#pragma unroll
            for (int r = 0; r < 4; ++r) tot[i][j][r] = fmaf(we, acc[i][j][r], tot[i][j][r]);
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
      }
    }
  }

  const int g = lane >> 4;
  if (a.split == 1) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = o0 + 32 * wo + 16 * i + 4 * g + r;
        if (o >= d_out) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int c = i0 + 32 * wi + 16 * j + lr;
          if (c < d_in) Lr.U[(long long)o * d_in + c] = tot[i][j][r];
        }
      }
  } else {
    float* P = a.partial + (long long)item * (kFO * kFI);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 2; ++j) P[(32 * wo + 16 * i + 4 * g + r) * kFI + 32 * wi + 16 * j + lr] = tot[i][j][r];
  }
}

// U = sum over splits of the partial tiles, in split order
__global__ __launch_bounds__(256) void update_reduce_kernel(UpdArgs a, int TO, int TI) {
  const int tile = blockIdx.y;
  int layer = 0;
  while (layer + 1 < a.num_layers && a.L[layer + 1].tile0 <= tile) ++layer;
  const UpdLayerArg& Lr = a.L[layer];
  const int t = tile - Lr.tile0, to = t / Lr.ti, ti = t - to * Lr.ti;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= TO * TI) return;
  const int o = to * TO + e / TI, c = ti * TI + e % TI;
  if (o >= Lr.d_out || c >= Lr.d_in) return;
  const float* P = a.partial + (long long)tile * a.split * (TO * TI) + e;
  float v = 0.f;
  for (int s = 0; s < a.split; ++s) v += P[(long long)s * (TO * TI)];
  Lr.U[(long long)o * Lr.d_in + c] = v;
}

// ------------------------------------------------------------------ host

struct UpdPlan {
  int64_t tiles;     // all layers
  int split;
  size_t off_ex, off_len, off_w, off_uex, off_ulen, off_uw, off_cnt, off_partial, bytes;
};

int cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus < 1)
    cus = 256;
  return cus;
}

void tile_dims(dr_dtype dtype, int& TO, int& TI) {
  TO = dtype == DR_BF16 ? kBO : kFO;
  TI = dtype == DR_BF16 ? kBI : kFI;
}

UpdPlan update_plan(const dr_layer* layers, int num_layers, int64_t n, dr_dtype dtype) {
  UpdPlan p;
  int TO, TI;
  tile_dims(dtype, TO, TI);
  p.tiles = 0;
  for (int l = 0; l < num_layers; ++l)
    p.tiles += ((layers[l].d_out + TO - 1) / TO) * ((layers[l].d_in + TI - 1) / TI);
  // resident workgroups: one bf16 workgroup (128 KB of LDS, 8 waves) or
  // four f32 workgroups per CU
  const int64_t slots = (int64_t)cu_count() * (dtype == DR_BF16 ? 1 : 4);
  int64_t split = 1;
  if (p.tiles < slots && n > 1) {
    split = (slots + p.tiles - 1) / p.tiles;
    if (split > kMaxSplit) split = kMaxSplit;
    if (split > n) split = n;
  }
  p.split = (int)split;
  const size_t nn = (size_t)(n > 0 ? n : 1) * num_layers;
  size_t o = 0;
  p.off_ex = o;      o = align_up(o + nn * 4, 256);
  p.off_len = o;     o = align_up(o + nn * 4, 256);
  p.off_w = o;       o = align_up(o + nn * 4, 256);
  p.off_uex = o;     o = align_up(o + nn * 4, 256);
  p.off_ulen = o;    o = align_up(o + nn * 4, 256);
  p.off_uw = o;      o = align_up(o + nn * 4, 256);
  p.off_cnt = o;     o = align_up(o + (size_t)num_layers * 4, 256);
  p.off_partial = o;
  if (p.split > 1) o = align_up(o + (size_t)p.tiles * p.split * TO * TI * 4, 256);
  p.bytes = o;
  return p;
}

dr_status validate_update(const dr_layer* layers, int num_layers, int64_t n, int64_t T, dr_dtype dtype,
                          const float* w, int P, int64_t ldw, const int32_t* group_of_layer, const float* U,
                          const int64_t* u_offset) {
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (!layers || num_layers < 1 || n < 0 || T < 0 || P < 1) return DR_ERR_ARG;
  if (n > (1 << 24) || T > (1 << 24) || ldw < n) return DR_ERR_ARG;
  if (n > 0 && !w) return DR_ERR_ARG;
  if (!U || !u_offset) return DR_ERR_ARG;
  const int64_t vec = dtype == DR_BF16 ? 8 : 4;
  const int64_t es = dtype == DR_BF16 ? 2 : 4;
  for (int l = 0; l < num_layers; ++l) {
    const dr_layer& L = layers[l];
    if (group_of_layer && (group_of_layer[l] < 0 || group_of_layer[l] >= P)) return DR_ERR_ARG;
    if (u_offset[l] < 0) return DR_ERR_ARG;
    if (L.d_in < 1 || L.d_out < 1 || L.d_in % vec || L.d_out % vec) return DR_ERR_ARG;
    if (L.d_in > (1 << 28) || L.d_out > (1 << 28)) return DR_ERR_ARG;
    if (L.ldx < L.d_in || L.lddy < L.d_out || L.ldx % vec || L.lddy % vec) return DR_ERR_ARG;
    if (n > 0 && T > 0) {
      if (!L.x || !L.dy || !aligned16(L.x) || !aligned16(L.dy)) return DR_ERR_ARG;
      // token rows are addressed with 32-bit offsets inside one example
      if (T * L.ldx * es >= (int64_t)kOobOffset - 64 || T * L.lddy * es >= (int64_t)kOobOffset - 64)
        return DR_ERR_UNSUPPORTED;
    }
  }
  return DR_OK;
}

__global__ void fill_f32_kernel(float* p, long long n, float v) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// s[i] = sum over the layer's tiles of the partial scores (tile order), 0 for empty examples
__global__ void direct_reduce_kernel(const double* part, int tiles, int n, const int* len, int T, float* s) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int L = len ? len[i] : T;
  L = L < 0 ? 0 : (L > T ? T : L);
  double t = 0.0;
  if (L > 0)
    for (int q = 0; q < tiles; ++q) t += part[(long long)q * n + i];
  s[i] = (float)t;
}

}  // namespace

size_t direct_workspace(const dr_layer* layers, int num_layers, int64_t n) {
  const UpdPlan pl = update_plan(layers, num_layers, n, DR_BF16);
  size_t o = align_up(pl.bytes, 256);
  o = align_up(o + (size_t)(n > 0 ? n : 1) * 4, 256);   // unit weights
  for (int l = 0; l < num_layers; ++l) {
    const int64_t tiles = ((layers[l].d_out + kBO - 1) / kBO) * ((layers[l].d_in + kBI - 1) / kBI);
    o = align_up(o + (size_t)tiles * (size_t)(n > 0 ? n : 1) * 8, 256);
  }
  return o;
}

// Direct scores s[l][i] = <gstar_l, G_i^(l)> of the first n examples, for
// bf16 layers whose target-mean gradients sit at gstar + g_off[l]
dr_status direct_scores(const dr_layer* layers, int num_layers, int64_t n, int64_t T, const int32_t* len,
                        const float* gstar, const int64_t* g_off, float* s, void* workspace, hipStream_t hs) {
  const UpdPlan pl = update_plan(layers, num_layers, n, DR_BF16);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  size_t o = align_up(pl.bytes, 256);
  float* ones = reinterpret_cast<float*>(ws + o);
  o = align_up(o + (size_t)(n > 0 ? n : 1) * 4, 256);
  double* part0 = reinterpret_cast<double*>(ws + o);
  if (n == 0) return DR_OK;
  hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, hs, ones, (long long)n, 1.0f);
  dr_status st = launch_status();
  UpdArgs base = {};
  base.split = pl.split;
  base.n = (int)n;
  base.nw = (int)n;
  base.ex = reinterpret_cast<const int*>(ws + pl.off_ex);
  base.exlen = reinterpret_cast<const int*>(ws + pl.off_len);
  base.exw = reinterpret_cast<const float*>(ws + pl.off_w);
  base.uex = reinterpret_cast<int*>(ws + pl.off_uex);
  base.ulen = reinterpret_cast<int*>(ws + pl.off_ulen);
  base.uw = reinterpret_cast<float*>(ws + pl.off_uw);
  base.cnt = reinterpret_cast<const int*>(ws + pl.off_cnt);
  base.partial = reinterpret_cast<float*>(ws + pl.off_partial);
  RowSel rs = {};
  if (st == DR_OK) {
    hipLaunchKernelGGL(update_plan_kernel, dim3(1), dim3(1024), 0, hs, (const float*)ones, (long long)n, base, len,
                       (int)T, 0, rs);
    st = launch_status();
  }
  if (st == DR_OK) {
    hipLaunchKernelGGL(update_sort_kernel, dim3((unsigned)((n + 255) / 256), 1), dim3(256), 0, hs, base);
    st = launch_status();
  }
  double* part = part0;
  for (int first = 0; first < num_layers && st == DR_OK; first += kMaxUpdLayers) {
    const int count = num_layers - first < kMaxUpdLayers ? num_layers - first : kMaxUpdLayers;
    UpdArgs a = base;
    int tiles = 0;
    double* parts[kMaxUpdLayers];
    int ltiles[kMaxUpdLayers];
    for (int j = 0; j < count; ++j) {
      const dr_layer& L = layers[first + j];
      UpdLayerArg& la = a.L[j];
      la.x = static_cast<const unsigned char*>(L.x);
      la.dy = static_cast<const unsigned char*>(L.dy);
      la.ldx = L.ldx;
      la.lddy = L.lddy;
      la.exx = T * L.ldx * 2;
      la.exdy = T * L.lddy * 2;
      la.d_in = (int)L.d_in;
      la.d_out = (int)L.d_out;
      la.ti = (int)((L.d_in + kBI - 1) / kBI);
      la.tile0 = tiles;
      la.list = 0;
      la.U = nullptr;
      la.gstar = gstar + g_off[first + j];
      la.part = part;
      ltiles[j] = (int)(((L.d_out + kBO - 1) / kBO) * la.ti);
      parts[j] = part;
      part = reinterpret_cast<double*>(reinterpret_cast<unsigned char*>(part) +
                                       align_up((size_t)ltiles[j] * (size_t)n * 8, 256));
      tiles += ltiles[j];
    }
    a.num_layers = count;
    a.ntiles = tiles;
    const int items = tiles * pl.split;
    hipLaunchKernelGGL(update_bf16_kernel<true>, dim3((items + 7) / 8 * 8), dim3(kBThreads), 0, hs, a);
    if ((st = launch_status()) != DR_OK) break;
    for (int j = 0; j < count && st == DR_OK; ++j) {
      hipLaunchKernelGGL(direct_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, hs,
                         (const double*)parts[j], ltiles[j], (int)n, len, (int)T, s + (long long)(first + j) * n);
      st = launch_status();
    }
  }
  return st;
}

namespace {
}  // namespace
}  // namespace dr

extern "C" size_t dr_update_workspace_size(const dr_layer* layers, int num_layers, int64_t n, int64_t T,
                                           dr_dtype dtype) {
  (void)T;
  if (!layers || num_layers < 1 || n < 0) return 0;
  if (dtype != DR_BF16 && dtype != DR_F32) return 0;
  for (int l = 0; l < num_layers; ++l)
    if (layers[l].d_in < 1 || layers[l].d_out < 1) return 0;
  return dr::update_plan(layers, num_layers, n, dtype).bytes;
}

extern "C" dr_status dr_assemble_update(const dr_layer* layers, int num_layers, int64_t n, int64_t T,
                                        const int32_t* len, dr_dtype dtype, const float* w, int P, int64_t ldw,
                                        const int32_t* group_of_layer, float* U, const int64_t* u_offset,
                                        void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  dr_status st = validate_update(layers, num_layers, n, T, dtype, w, P, ldw, group_of_layer, U, u_offset);
  if (st != DR_OK) return st;
  const UpdPlan pl = update_plan(layers, num_layers, n, dtype);
  if (!workspace || ws_bytes < pl.bytes) return DR_ERR_WORKSPACE;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  int TO, TI;
  tile_dims(dtype, TO, TI);
  const int64_t es = dtype == DR_BF16 ? 2 : 4;
  const int nstride = n > 0 ? (int)n : 1;
  // one example list per distinct weight row, in order of first use
  int* layer_list = new int[num_layers];
  int* list_row = new int[num_layers];
  int nlists = 0;
  for (int l = 0; l < num_layers; ++l) {
    const int row = group_of_layer ? group_of_layer[l] : 0;
    int q = 0;
    while (q < nlists && list_row[q] != row) ++q;
    if (q == nlists) list_row[nlists++] = row;
    layer_list[l] = q;
  }
  UpdArgs base = {};
  base.split = pl.split;
  base.n = nstride;
  base.nw = (int)n;
  base.ex = reinterpret_cast<const int*>(ws + pl.off_ex);
  base.exlen = reinterpret_cast<const int*>(ws + pl.off_len);
  base.exw = reinterpret_cast<const float*>(ws + pl.off_w);
  base.uex = reinterpret_cast<int*>(ws + pl.off_uex);
  base.ulen = reinterpret_cast<int*>(ws + pl.off_ulen);
  base.uw = reinterpret_cast<float*>(ws + pl.off_uw);
  base.cnt = reinterpret_cast<const int*>(ws + pl.off_cnt);
  base.partial = reinterpret_cast<float*>(ws + pl.off_partial);
  for (int first = 0; first < nlists && st == DR_OK; first += kMaxUpdLayers) {
    const int count = nlists - first < kMaxUpdLayers ? nlists - first : kMaxUpdLayers;
    RowSel rs;
    for (int j = 0; j < kMaxUpdLayers; ++j) rs.r[j] = j < count ? list_row[first + j] : 0;
    hipLaunchKernelGGL(update_plan_kernel, dim3(count), dim3(1024), 0, hs, w, (long long)ldw, base, len, (int)T,
                       first, rs);
    st = launch_status();
  }
  if (st == DR_OK && n > 0) {
    hipLaunchKernelGGL(update_sort_kernel, dim3((unsigned)((n + 255) / 256), nlists), dim3(256), 0, hs, base);
    st = launch_status();
  }
  for (int first = 0; first < num_layers && st == DR_OK; first += kMaxUpdLayers) {
    const int count = num_layers - first < kMaxUpdLayers ? num_layers - first : kMaxUpdLayers;
    UpdArgs a = base;
    int tiles = 0;
    for (int j = 0; j < count; ++j) {
      const dr_layer& L = layers[first + j];
      UpdLayerArg& la = a.L[j];
      la.x = static_cast<const unsigned char*>(L.x);
      la.dy = static_cast<const unsigned char*>(L.dy);
      la.ldx = L.ldx;
      la.lddy = L.lddy;
      la.exx = T * L.ldx * es;
      la.exdy = T * L.lddy * es;
      la.d_in = (int)L.d_in;
      la.d_out = (int)L.d_out;
      la.ti = (int)((L.d_in + TI - 1) / TI);
      la.tile0 = tiles;
      la.list = layer_list[first + j];
      la.U = U + u_offset[first + j];
      tiles += (int)(((L.d_out + TO - 1) / TO) * la.ti);
    }
    a.num_layers = count;
    a.ntiles = tiles;
    const int items = tiles * pl.split;
    const int grid = (items + 7) / 8 * 8;
    if (dtype == DR_BF16)
      hipLaunchKernelGGL(update_bf16_kernel<false>, dim3(grid), dim3(kBThreads), 0, hs, a);
    else
      hipLaunchKernelGGL(update_f32_kernel, dim3(grid), dim3(kFThreads), 0, hs, a);
    if ((st = launch_status()) != DR_OK) break;
    if (pl.split > 1) {
      hipLaunchKernelGGL(update_reduce_kernel, dim3((TO * TI + 255) / 256, tiles), dim3(256), 0, hs, a, TO, TI);
      st = launch_status();
    }
  }
  delete[] layer_list;
  delete[] list_row;
  return st;
}
