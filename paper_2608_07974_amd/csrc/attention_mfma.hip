// MFMA flash attention for bf16, head_dim 64 or 128 (the decoder layers of
// f_k in Eq. (1)): causal, GQA (q-head h reads kv-head h / (Hq / Hkv)),
// right padding by seq_len, scores q.k / sqrt(hd), fp32 softmax statistics.
//
// MFMA 16x16x32 bf16.  Lane l of a wave: c = l % 16 (output column), g = l / 16.
// A and B operands only have to agree on which 8 reduction indices each lane
// group carries; here that set is {32kk + 4g + r} and {32kk + 16 + 4g + r},
// r < 4, which is exactly how the C layout of a 16-row MFMA block hands out
// rows (4g + r) -- so softmax probabilities feed the next MFMA straight from
// registers.
//  - Forward: each wave owns 2 x 16 queries; S^T = K Q^T puts one query per
//    lane column, so the online-softmax statistics live per lane, and
//    O^T += V^T P^T reads V^T with the LDS transpose read.
//  - dK/dV: one workgroup per (128 keys, kv-head), walking every q-head of
//    its group and every later query tile (no cross-workgroup reduction).
//  - dQ: one workgroup per (128 queries, q-head).
// Tiles of 64 rows are copied global -> LDS by the buffer unit
// (buffer_load ... lds, no staging registers) into double-buffered LDS,
// 16-byte chunks XOR-swizzled by row, so the copies overlap the MFMAs.
// Operands needed transposed are read from the same row-major tiles with
// ds_read_b64_tr_b16: within each 16-lane group, lane r addresses row
// q0 + r/4, columns d0 + 4 (r % 4) .. +3, and lane i receives column d0 + i
// of rows q0 .. q0 + 3.
#include "common.h"

namespace zl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));

namespace {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int BT = 64;   // rows of a staged tile
constexpr int BW = 128;  // rows (queries or keys) owned by a workgroup: 4 waves x 32
constexpr int NTH = 256;

__device__ inline f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// XOR permutation of a row's 16-byte chunks in LDS.  Two read shapes use a
// tile: row fragments (16 bytes per lane, rows 16m + c, chunk 4kk + g for
// lane 16g + c) and transposed column fragments (ds_read_b64_tr_b16, 8 rows
// per half-wave, two adjacent chunks per row).  Measured on gfx950: a 16-byte
// read serves in one cycle the 16 lanes that share lane bit 5 and the parity
// of lane bits 2-4, and a transpose read a half-wave.  Both are then free of
// bank conflicts when, at 256-byte rows (head size 128), the permutation
// shifted left by one keeps a half-wave's 8 rows in distinct 32-byte groups
// and x -> swz(x) ^ (bit 2 ^ bit 3 of x) stays one-to-one on 16 rows:
// `(row & 7) << 1`.  `row & 15` cost the transpose reads a 2-way conflict.
// At 128-byte rows (head size 64), `row & 7` meets both.
template <int HD>
__device__ inline int swz(int row) {
  return HD == 128 ? ((row & 7) << 1) : (row & 7);
}

__device__ inline bf16x8_t zero8() {
  return __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
}

__device__ inline __bf16 to_bf16(float f) { return __builtin_bit_cast(__bf16, f32_to_bf16(f)); }

// Max over lanes l and l ^ 16 (l ^ 32): the permlane swaps exchange 16-lane
// rows (32-lane halves) of two copies of x, so each lane ends up holding its
// own value and its partner's in the two results (VALU, no LDS round trip).
__device__ inline float max_xor16(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, r[0]), __builtin_bit_cast(float, r[1]));
}
__device__ inline float max_xor32(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, r[0]), __builtin_bit_cast(float, r[1]));
}

// 8 consecutive bf16 of row `row`, 16-byte chunk `ch`.
template <int HD>
__device__ inline bf16x8_t frag_row(const bf16_t* lds, int row, int ch) {
  return *reinterpret_cast<const bf16x8_t*>(lds + row * HD + ((ch ^ swz<HD>(row)) * 8));
}

// Column d0 + c of rows {rb + 4g + k} then {rb + 16 + 4g + k}, k < 4 (the k-set
// of lane group g), through the LDS transpose read.
template <int HD>
__device__ inline bf16x8_t frag_col(const bf16_t* lds, int rb, int g, int d0, int c) {
  const int r1 = rb + 4 * g + (c >> 2), r2 = r1 + 16;
  const int col = d0 + 4 * (c & 3);
  const bf16_t* p1 = lds + r1 * HD + (((col >> 3) ^ swz<HD>(r1)) << 3) + (col & 7);
  const bf16_t* p2 = lds + r2 * HD + (((col >> 3) ^ swz<HD>(r2)) << 3) + (col & 7);
  const s16x4_t x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4_t*)(p1));
  const s16x4_t y = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4_t*)(p2));
  const s16x8_t xy = __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8_t, xy);
}

// Inverse (transposed) rotate-half RoPE of one row held as HD/16 register
// blocks x[db][r] (dims 16*db + c): pairs (j, j + HD/2) sit HD/32 blocks
// apart in the same lane.  du_j = du'_j c + du'_{j+h} s,
// du_{j+h} = du'_{j+h} c - du'_j s.
template <int HD>
__device__ inline void rope_back(f32x4_t (&x)[HD / 16], int r, const int32_t* pos, int64_t row,
                                 const float2* table, int max_pos, int c) {
  int p = pos[row];
  p = p < 0 ? 0 : (p >= max_pos ? max_pos - 1 : p);
  constexpr int HB = HD / 32;
#pragma unroll
  for (int db = 0; db < HB; ++db) {
    const float2 cs = table[(int64_t)p * (HD / 2) + db * 16 + c];
    const float a = x[db][r], b = x[db + HB][r];
    x[db][r] = a * cs.x + b * cs.y;
    x[db + HB][r] = b * cs.x - a * cs.y;
  }
}

}  // namespace

// ------------------------------------------------------ direct-to-LDS copy
// Tiles of BT rows x HD are copied global -> LDS by the buffer unit (16 bytes
// per lane; lane i's bytes land at M0 + 16 i; offsets at or above the record
// count read as zero), into the same row-major, chunk-swizzled layout the
// fragment readers use.
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
constexpr uint32_t DMA_OOB = 0x80000000u;

__device__ inline i32x4_t buffer_rsrc(const void* base) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  i32x4_t r;
  r[0] = (int32_t)(uint32_t)p;
  r[1] = (int32_t)(uint32_t)(p >> 32);
  r[2] = (int32_t)DMA_OOB;
  r[3] = 0x00020000;
  return r;
}
// The copies carry no compiler memory clobber: their ordering against the
// LDS reads of a stage comes from the workgroup barriers and the explicit
// vmcnt waits around them (a clobber only kept the compiler from
// scheduling other memory operations across the copies: 1 % slower).
__device__ inline void dma16(uint32_t lds_byte, uint32_t voff, i32x4_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_byte), "v"(voff), "s"(rsrc));
}
__device__ inline void dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// 4 bytes per lane: lane i's dword lands at M0 + 4 i
__device__ inline void dma4(uint32_t lds_byte, uint32_t voff, i32x4_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(lds_byte), "v"(voff), "s"(rsrc));
}
// A resource of `bytes` bytes: offsets at or past it read as zero.
__device__ inline i32x4_t buffer_rsrc_n(const void* base, uint32_t bytes) {
  i32x4_t r = buffer_rsrc(base);
  r[2] = (int32_t)bytes;
  return r;
}
// s_waitcnt vmcnt(N), other counters unconstrained (gfx9 encoding)
template <int N>
__device__ inline void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// This wave's copies of the oldest outstanding tile have landed once at
// most `ahead` later tiles' copies (PER instructions each) are in flight.
template <int PER>
__device__ inline void wait_tiles(int ahead) {
  if (ahead >= 2) wait_vm<2 * PER>();
  else if (ahead == 1) wait_vm<PER>();
  else wait_vm<0>();
}

template <int HD, int NT, int ROWS = BT>
struct TileDma {
  static constexpr int CH = HD / 8;              // 16-byte chunks per row
  static constexpr int RPI = 64 / CH;            // rows per copy instruction
  static constexpr int ITEMS = ROWS * CH / NT;   // chunks per thread
  static_assert(ITEMS >= 1 && ITEMS * NT == ROWS * CH, "tile chunks must divide over the threads");
  int rl, cl;       // lane's row within an instruction's rows, and its chunk
  uint32_t ldb;     // bytes per matrix row
  __device__ inline void init(int lane, int64_t ld) {
    rl = lane / CH;
    cl = lane % CH;
    ldb = (uint32_t)ld * 2u;
  }
  // rows r0 .. r0+ROWS-1 of the matrix (rows >= rvalid read as zero)
  __device__ inline void issue(uint32_t lds_byte, int wave, int r0, int rvalid, i32x4_t rsrc) const {
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      const int row = (wave * ITEMS + j) * RPI + rl;  // tile row this lane's chunk lands in
      const int ch = cl ^ swz<HD>(row);               // source chunk for that LDS slot
      const uint32_t v = r0 + row < rvalid ? (uint32_t)(r0 + row) * ldb + (uint32_t)ch * 16u : DMA_OOB;
      dma16(lds_byte + (uint32_t)(wave * ITEMS + j) * 1024u, v, rsrc);
    }
  }
};

// ------------------------------------------------------- workgroup order
// Causal work per workgroup grows (forward, dQ) or shrinks (dK/dV) with the
// x index of the grid, and workgroups are dispatched with x varying
// fastest.  Reading the linear dispatch index as (x slowest, then y, then
// z) starts the longest blocks of every (batch, head group) first, which
// keeps the last wave of the launch short (longest-first list scheduling).
struct CausalOrder {
  int x, y, z;
};
__device__ inline CausalOrder causal_order() {
  const int nyz = gridDim.y * gridDim.z;
  const int lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int r = lin % nyz;
  return CausalOrder{lin / nyz, r % (int)gridDim.y, r / (int)gridDim.y};
}

// ------------------------------------------------------------------ forward
// Workgroup: 8 waves; HPW q-heads of one kv group (they share every K/V
// tile) x 256 / HPW queries; each wave owns 32 queries of one head.
// Online softmax in the log2 domain with a lazily moved reference maximum:
// a row's reference only moves when the running maximum exceeds it by more
// than 8 (probabilities stay <= 2^8, exact after the final division), so
// the O rescale is skipped on most tiles.  Causal/length masks are applied
// only on tiles that cross the diagonal or the end of the keys.
constexpr int FW_WAVES = 8;
constexpr int FW_NT = FW_WAVES * 64;
#ifndef FW_NST
#define FW_NST 2  // K/V tile stages of the forward and dQ kernels (3: slower)
#endif
static_assert(FW_NST >= 2 && FW_NST <= 4, "K/V pipeline depth");
constexpr float RESCALE_TAU = 8.f;

template <int HD, int HPW>
__global__ void __launch_bounds__(FW_NT) attn_fwd_mfma(AttnDesc a) {
  constexpr int QW = FW_WAVES / HPW;   // query sub-blocks of 32 per head
  constexpr int QB = QW * 32;          // queries per workgroup
  constexpr uint32_t TB = BT * HD * 2; // bytes of one K or V tile
  extern __shared__ __align__(16) unsigned char smem[];
  const CausalOrder co = causal_order();
  const int qb = gridDim.x - 1 - co.x;  // longest causal rows first
  const int hb = co.y * HPW, b = co.z;
  const int kvh = hb / (a.Hq / a.Hkv);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int c = lane & 15, g = lane >> 4;
  const int h = hb + wave % HPW;
  const int q0 = qb * QB, qw0 = q0 + (wave / HPW) * 32;
  const int L = a.seq_lens[b];
  const int64_t rowb = (int64_t)b * a.S;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q);
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k);
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v);

  int qi[2];
  bf16x8_t qf[2][HD / 32];
  f32x4_t o[2][HD / 16];
  float m[2], lsum[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    qi[j] = qw0 + j * 16 + c;
#pragma unroll
    for (int kk = 0; kk < HD / 32; ++kk)
      qf[j][kk] = qi[j] < a.S ? *reinterpret_cast<const bf16x8_t*>(Q + (rowb + qi[j]) * a.ldq +
                                                                   (int64_t)h * HD + 8 * g + 32 * kk)
                              : zero8();
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) o[j][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m[j] = -INFINITY;
    lsum[j] = 0.f;
  }
  const float cs = a.scale * LOG2E;
  const int kend = min(min(q0 + QB, a.S), L);        // keys any query here may see
  const int kend_w = min(min(qw0 + 32, a.S), L);     // keys this wave's queries may see
  const int nt = (kend + BT - 1) / BT;

  const i32x4_t rk = buffer_rsrc(K + rowb * a.ldk + (int64_t)kvh * HD);
  const i32x4_t rv = buffer_rsrc(V + rowb * a.ldv + (int64_t)kvh * HD);
  TileDma<HD, FW_NT> dk, dv;
  dk.init(lane, a.ldk);
  dv.init(lane, a.ldv);
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(smem);  // [FW_NST][K | V]
  // K/V tile t goes to stage t % FW_NST, FW_NST - 1 tiles ahead of its use
  for (int p = 0; p < FW_NST - 1 && p < nt; ++p) {
    dk.issue(lds0 + p * 2 * TB, wave, p * BT, kend, rk);
    dv.issue(lds0 + p * 2 * TB + TB, wave, p * BT, kend, rv);
  }
  int rd = 0, wr = FW_NST - 1;
  for (int t = 0; t < nt; ++t) {
    const int k0 = t * BT;
    wait_tiles<2 * TileDma<HD, FW_NT>::ITEMS>(min(FW_NST - 2, nt - 1 - t));
    __syncthreads();  // tile t everywhere; stage wr (tile t - 1) is no longer read
    if (t + FW_NST - 1 < nt) {
      dk.issue(lds0 + wr * 2 * TB, wave, (t + FW_NST - 1) * BT, kend, rk);
      dv.issue(lds0 + wr * 2 * TB + TB, wave, (t + FW_NST - 1) * BT, kend, rv);
    }
    const bf16_t* kt = reinterpret_cast<const bf16_t*>(smem + rd * 2 * TB);
    rd = rd + 1 == FW_NST ? 0 : rd + 1;
    wr = wr + 1 == FW_NST ? 0 : wr + 1;
    if (k0 >= kend_w) continue;  // past every key this wave's queries see
    const bf16_t* vt = kt + BT * HD;
    // S^T: 8 independent accumulators per k-step; the K fragments of the
    // k-step two ahead are read while the current step's MFMAs run
    constexpr int NK = HD / 32, KA = NK < 3 ? NK : 3;
    f32x4_t s[2][4];
    bf16x8_t kb[KA][4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      s[0][blk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      s[1][blk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int kk = 0; kk < KA - 1; ++kk)
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) kb[kk][blk] = frag_row<HD>(kt, blk * 16 + c, g + 4 * kk);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      const int cur = kk % KA;
      if (kk + KA - 1 < NK) {
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
          kb[(kk + KA - 1) % KA][blk] = frag_row<HD>(kt, blk * 16 + c, g + 4 * (kk + KA - 1));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) {
        s[0][blk] = mfma16(kb[cur][blk], qf[0][kk], s[0][blk]);
        s[1][blk] = mfma16(kb[cur][blk], qf[1][kk], s[1][blk]);
      }
    }
    // V^T fragments of the O update: a ring of VA reads in flight, the first
    // VA issued before the softmax so that it hides their latency
    constexpr int NV = 2 * (HD / 16), VA = 4;
    bf16x8_t vb[VA];
#pragma unroll
    for (int i = 0; i < VA; ++i) vb[i] = frag_col<HD>(vt, 32 * (i & 1), g, 16 * (i >> 1), c);
    // some key of the tile lies after some query of the wave, or past kend
    const bool masked = k0 + BT - 1 > qw0 || k0 + BT > kend;
    bf16x8_t pf[2][2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      // raw scores: the maximum is taken before scaling (cs > 0) and the
      // scale is folded into the exponent's FMA
      float x[4][4];
      float tmax = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
#pragma unroll
        for (int r = 0; r < 4; ++r) x[blk][r] = s[j][blk][r];
      if (masked) {
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = k0 + blk * 16 + 4 * g + r;
            x[blk][r] = (key <= qi[j] && key < kend) ? x[blk][r] : -INFINITY;
          }
      }
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
        tmax = fmaxf(tmax, fmaxf(fmaxf(x[blk][0], x[blk][1]), fmaxf(x[blk][2], x[blk][3])));
      tmax = max_xor32(max_xor16(tmax)) * cs;
      const bool move = tmax > m[j] + RESCALE_TAU;
      if (__any(move)) {
        const float mnew = move ? tmax : m[j];
        const float alpha = move ? (m[j] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[j] - mnew)) : 1.f;
        m[j] = mnew;
        lsum[j] *= alpha;
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) o[j][db] *= alpha;
      }
      const float nms = m[j] == -INFINITY ? 0.f : -m[j];
      float psum = 0.f;
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(x[blk][r], cs, nms));
          psum += p;
          pf[j][blk >> 1][(blk & 1) * 4 + r] = (__bf16)p;
        }
      lsum[j] += psum;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {  // i = 2 db + kk
      const int db = i >> 1, kk = i & 1, cur = i % VA;
      __builtin_amdgcn_sched_barrier(0);
      o[0][db] = mfma16(vb[cur], pf[0][kk], o[0][db]);
      o[1][db] = mfma16(vb[cur], pf[1][kk], o[1][db]);
      if (i + VA < NV) vb[cur] = frag_col<HD>(vt, 32 * ((i + VA) & 1), g, 16 * ((i + VA) >> 1), c);
    }
  }
  dma_wait();
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    float ls = lsum[j];
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    if (qi[j] < a.S) {
      const float inv = ls > 0.f ? 1.f / ls : 0.f;
      bf16_t* O = reinterpret_cast<bf16_t*>(a.o) + (rowb + qi[j]) * a.ldo + (int64_t)h * HD;
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        const ushort4 w = make_ushort4(f32_to_bf16(o[j][db][0] * inv), f32_to_bf16(o[j][db][1] * inv),
                                       f32_to_bf16(o[j][db][2] * inv), f32_to_bf16(o[j][db][3] * inv));
        *reinterpret_cast<ushort4*>(O + db * 16 + 4 * g) = w;
      }
      if (g == 0)
        a.lse[((int64_t)b * a.Hq + h) * a.S + qi[j]] = ls > 0.f ? m[j] * LN2 + __logf(ls) : -INFINITY;
    }
  }
}

// ------------------------------------------------------------------ delta
// delta[b, h, i] = sum_d dO[i, h, d] * O[i, h, d]; one wave per (row, head).
template <int HD>
__global__ void __launch_bounds__(256) attn_delta_mfma(AttnDesc a) {
  const int64_t w = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t n = (int64_t)a.B * a.Hq * a.S;
  if (w >= n) return;
  const int i = (int)(w % a.S);
  const int h = (int)((w / a.S) % a.Hq);
  const int b = (int)(w / ((int64_t)a.S * a.Hq));
  const int64_t row = (int64_t)b * a.S + i;
  const bf16_t* O = reinterpret_cast<const bf16_t*>(a.o) + row * a.ldo + (int64_t)h * HD;
  const bf16_t* D = reinterpret_cast<const bf16_t*>(a.dout) + row * a.lddo + (int64_t)h * HD;
  float s = 0.f;
  for (int d = lane; d < HD; d += 64) s += bf16_to_f32(O[d]) * bf16_to_f32(D[d]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) a.delta[((int64_t)b * a.Hq + h) * a.S + i] = s;
}

// ------------------------------------------------------------------- dK dV
// One workgroup per (KV_KB keys, kv-head): KV_WAVES waves (8) of 16 keys walk every
// (q-head, query tile) pair of the kv group; the pair's Q and dO tiles are
// copied direct-to-LDS once for all waves, KV_NST - 1 pairs ahead of use, with
// the pair's softmax statistics (lse, delta of its KV_BQ queries).  16 keys per wave keeps
// the K/V fragments and the fp32 dK/dV accumulators within two waves per
// SIMD.
#ifndef KV_WAVES
#define KV_WAVES 8
#endif
constexpr int KV_NT = KV_WAVES * 64;
constexpr int KV_KB = KV_WAVES * 16;  // keys per workgroup
#ifndef KV_NST
#define KV_NST 2
#endif
#ifndef DKV_CA
#define DKV_CA 3
#endif
#ifndef KV_BQ
#define KV_BQ 128  // queries per (q-head, query tile) pair (64: 2 % slower)
#endif
static_assert(KV_BQ % 64 == 0, "query tiles of whole 64-row copies");
template <int HD>
constexpr size_t dkv_lds_bytes() {  // KV_NST x (Q | dO tiles, lse | delta of KV_BQ queries)
  return (size_t)KV_NST * (2 * KV_BQ * HD * 2 + 2 * KV_BQ * 4);
}

template <int HD>
__global__ void __launch_bounds__(KV_NT, 2) attn_dkv_mfma(AttnDesc a) {
  constexpr int BQ = KV_BQ;
  constexpr uint32_t TB = BQ * HD * 2;     // one Q or dO tile
  constexpr uint32_t STAGE = 2 * TB + 2 * BQ * 4;  // Q | dO | lse | delta
  constexpr int NST = KV_NST;
  static_assert(NST >= 2 && NST <= 4 && NST * STAGE <= 160 * 1024, "pipeline depth");
  extern __shared__ __align__(16) unsigned char smem[];
  const CausalOrder co = causal_order();
  const int kblk = co.x;                   // early keys see the most queries: first
  const int kvh = co.y, b = co.z;
  const int grp = a.Hq / a.Hkv;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int c = lane & 15, g = lane >> 4;
  const int L = a.seq_lens[b];
  const int k0 = kblk * KV_KB;
  const int kw0 = k0 + wave * 16;
  const int klim = min(a.S, L);
  const int kj = kw0 + c;
  const int64_t rowb = (int64_t)b * a.S;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q);
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k);
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v);
  const bf16_t* DO = reinterpret_cast<const bf16_t*>(a.dout);

  bf16x8_t kf[HD / 32], vf[HD / 32];
  f32x4_t dk[HD / 16], dv[HD / 16];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk) {
    const int64_t off = (int64_t)kvh * HD + 8 * g + 32 * kk;
    kf[kk] = kj < klim ? *reinterpret_cast<const bf16x8_t*>(K + (rowb + kj) * a.ldk + off) : zero8();
    vf[kk] = kj < klim ? *reinterpret_cast<const bf16x8_t*>(V + (rowb + kj) * a.ldv + off) : zero8();
  }
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) {
    dk[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    dv[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const float cs = a.scale * LOG2E;
  // (q-head, query tile) pairs; a key block's query tiles start at k0
  const int ntq = k0 < klim ? (a.S - k0 + BQ - 1) / BQ : 0;
  const int npair = grp * ntq;

  TileDma<HD, KV_NT, BQ> dq_, dd_;
  dq_.init(lane, a.ldq);
  dd_.init(lane, a.lddo);
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(smem);
  const int64_t so_b = (int64_t)b * a.Hq * a.S;
  // Copies of pair pr into stage pr % NST: the Q and dO tiles (every wave
  // its share) and, by wave 0, the pair's lse and delta rows (one dword per
  // lane; queries past S read as zero)
  constexpr int PER = 2 * TileDma<HD, KV_NT, BQ>::ITEMS;  // tile copies per wave and pair
  constexpr int PST = 2 * (BQ / 64);                      // wave 0's statistics copies
  auto issue = [&](int pr, int stage) {
    const int h = kvh * grp + pr / ntq;
    const int q0 = k0 + (pr % ntq) * BQ;
    const uint32_t dst = lds0 + (uint32_t)stage * STAGE;
    dq_.issue(dst, wave, q0, a.S, buffer_rsrc(Q + rowb * a.ldq + (int64_t)h * HD));
    dd_.issue(dst + TB, wave, q0, a.S, buffer_rsrc(DO + rowb * a.lddo + (int64_t)h * HD));
    if (wave == 0) {
      const int64_t so = so_b + (int64_t)h * a.S;
      const uint32_t bytes = (uint32_t)a.S * 4u;
#pragma unroll
      for (int i = 0; i < BQ / 64; ++i) {
        const uint32_t vo = (uint32_t)(q0 + 64 * i + lane) * 4u;
        dma4(dst + 2 * TB + 256 * i, vo, buffer_rsrc_n(a.lse + so, bytes));
        dma4(dst + 2 * TB + BQ * 4 + 256 * i, vo, buffer_rsrc_n(a.delta + so, bytes));
      }
    }
  };
  // this wave's copies of pair pr have landed once at most `ahead` later
  // pairs' copies are still outstanding
  auto wait_pair = [&](int ahead) {
    if (wave == 0) {
      if (ahead >= 2) wait_vm<2 * (PER + PST)>();
      else if (ahead == 1) wait_vm<PER + PST>();
      else wait_vm<0>();
    } else {
      if (ahead >= 2) wait_vm<2 * PER>();
      else if (ahead == 1) wait_vm<PER>();
      else wait_vm<0>();
    }
  };
  static_assert(2 * (PER + PST) < 64, "vmcnt range");
  for (int p = 0; p < NST - 1 && p < npair; ++p) issue(p, p);
  int rd = 0, wr = NST - 1;  // stage read by pair pr, stage written for pair pr + NST - 1
#pragma unroll 1
  for (int pr = 0; pr < npair; ++pr) {
    wait_pair(min(NST - 2, npair - 1 - pr));
    __syncthreads();  // pair pr's copies everywhere; stage wr (read by pair pr - 1) is free
    if (pr + NST - 1 < npair) issue(pr + NST - 1, wr);
    const int q0 = k0 + (pr % ntq) * BQ;
    const unsigned char* sb = smem + rd * STAGE;
    rd = rd + 1 == NST ? 0 : rd + 1;
    wr = wr + 1 == NST ? 0 : wr + 1;
    const bf16_t* qt = reinterpret_cast<const bf16_t*>(sb);
    const bf16_t* dt = qt + BQ * HD;
    const float* lss = reinterpret_cast<const float*>(sb + 2 * TB);  // lse (natural log)
    const float* dls = lss + BQ;
    // some key of the wave lies after some query of the tile, or keys or
    // queries run past their ends (every query before S sees key 0, so its
    // lse is finite; queries past S read lse = 0 and are masked)
    const bool masked = kw0 + 15 > q0 || q0 + BQ > a.S || kw0 + 16 > klim;
    // Fragment reads run ahead of the MFMAs that use them: the Q / dO row
    // fragments of the next 16-query block (double-buffered), and the
    // transposed dO / Q column fragments of the dV / dK update (a ring of
    // DKV_CA reads in flight).
    bf16x8_t fq[2][HD / 32], fd[2][HD / 32];
#pragma unroll
    for (int kk = 0; kk < HD / 32; ++kk) {
      fq[0][kk] = frag_row<HD>(qt, c, g + 4 * kk);
      fd[0][kk] = frag_row<HD>(dt, c, g + 4 * kk);
    }
#pragma unroll
    for (int half = 0; half < BQ / 32; ++half) {
      bf16x8_t pk, dsk;
#pragma unroll
      for (int qq = 0; qq < 2; ++qq) {
        const int qb = 2 * half + qq, cur = qb & 1;
        if (qb + 1 < BQ / 16) {
#pragma unroll
          for (int kk = 0; kk < HD / 32; ++kk) {
            fq[cur ^ 1][kk] = frag_row<HD>(qt, (qb + 1) * 16 + c, g + 4 * kk);
            fd[cur ^ 1][kk] = frag_row<HD>(dt, (qb + 1) * 16 + c, g + 4 * kk);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        // two independent accumulation chains, interleaved
        f32x4_t sc = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < HD / 32; ++kk) {
          sc = mfma16(fq[cur][kk], kf[kk], sc);
          dp = mfma16(fd[cur][kk], vf[kk], dp);
        }
        // the mask as one uniform branch over the block's four scores
        // (most pairs skip it), not a select per score
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) x[r] = sc[r] * cs - lss[qb * 16 + 4 * g + r] * LOG2E;
        if (masked) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int q = q0 + qb * 16 + 4 * g + r;
            x[r] = (kj <= q && q < a.S && kj < klim) ? x[r] : -INFINITY;
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(x[r]);
          pk[qq * 4 + r] = (__bf16)p;
          dsk[qq * 4 + r] = (__bf16)(p * (dp[r] - dls[qb * 16 + 4 * g + r]));
        }
      }
      // dV += P^T dO, dK += dS^T Q over this half's 32 queries
      // (transposed dO / Q column fragments: a ring of CA reads in flight)
      constexpr int NCOL = HD / 16, CA = DKV_CA;
      bf16x8_t dcol[CA], qcol[CA];
#pragma unroll
      for (int i = 0; i < CA; ++i) {
        dcol[i] = frag_col<HD>(dt, 32 * half, g, 16 * i, c);
        qcol[i] = frag_col<HD>(qt, 32 * half, g, 16 * i, c);
      }
#pragma unroll
      for (int db = 0; db < NCOL; ++db) {
        const int cur = db % CA;
        __builtin_amdgcn_sched_barrier(0);
        dv[db] = mfma16(pk, dcol[cur], dv[db]);
        dk[db] = mfma16(dsk, qcol[cur], dk[db]);
        if (db + CA < NCOL) {
          dcol[cur] = frag_col<HD>(dt, 32 * half, g, 16 * (db + CA), c);
          qcol[cur] = frag_col<HD>(qt, 32 * half, g, 16 * (db + CA), c);
        }
      }
    }
  }
  dma_wait();
  bf16_t* DK = reinterpret_cast<bf16_t*>(a.dk);
  bf16_t* DV = reinterpret_cast<bf16_t*>(a.dv);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int key = kw0 + 4 * g + r;
    if (key < a.S) {
      if (a.rope) rope_back<HD>(dk, r, a.pos, rowb + key, a.rope, a.max_pos, c);
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        const int64_t col = (int64_t)kvh * HD + db * 16 + c;
        DK[(rowb + key) * a.lddk + col] = f32_to_bf16(dk[db][r] * a.scale);
        DV[(rowb + key) * a.lddv + col] = f32_to_bf16(dv[db][r]);
      }
    }
  }
}

// ----------------------------------------------------------------------- dQ
// Same decomposition as the forward: 8 waves, HPW q-heads of one kv group
// share every K/V tile (direct-to-LDS copy); each wave owns 32 queries.
// dS = P (dP - delta) with P recomputed from the saved log-sum-exp; masks
// only on tiles crossing the diagonal or the end of the keys.
template <int HD, int HPW>
__global__ void __launch_bounds__(FW_NT) attn_dq_mfma(AttnDesc a) {
  constexpr int QW = FW_WAVES / HPW;
  constexpr int QB = QW * 32;
  constexpr uint32_t TB = BT * HD * 2;
  extern __shared__ __align__(16) unsigned char smem[];
  const CausalOrder co = causal_order();
  const int qblk = gridDim.x - 1 - co.x;
  const int hb = co.y * HPW, b = co.z;
  const int kvh = hb / (a.Hq / a.Hkv);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int c = lane & 15, g = lane >> 4;
  const int h = hb + wave % HPW;
  const int q0 = qblk * QB, qw0 = q0 + (wave / HPW) * 32;
  const int L = a.seq_lens[b];
  const int64_t rowb = (int64_t)b * a.S;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q);
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k);
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v);
  const bf16_t* DO = reinterpret_cast<const bf16_t*>(a.dout);

  int qi[2];
  bf16x8_t qf[2][HD / 32], df[2][HD / 32];
  float l2[2], dl[2];
  f32x4_t dq[2][HD / 16];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    qi[j] = qw0 + j * 16 + c;
    const bool ok = qi[j] < a.S;
#pragma unroll
    for (int kk = 0; kk < HD / 32; ++kk) {
      const int64_t col = (int64_t)h * HD + 8 * g + 32 * kk;
      qf[j][kk] = ok ? *reinterpret_cast<const bf16x8_t*>(Q + (rowb + qi[j]) * a.ldq + col) : zero8();
      df[j][kk] = ok ? *reinterpret_cast<const bf16x8_t*>(DO + (rowb + qi[j]) * a.lddo + col) : zero8();
    }
    const int64_t so = ((int64_t)b * a.Hq + h) * a.S + qi[j];
    const float lse = ok ? a.lse[so] : -INFINITY;
    // a query with no key (or outside the sequence) gets +inf: every p = 0
    l2[j] = lse == -INFINITY ? INFINITY : lse * LOG2E;
    dl[j] = ok ? a.delta[so] : 0.f;
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) dq[j][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const float cs = a.scale * LOG2E;
  const int kend = min(min(q0 + QB, a.S), L);
  const int kend_w = min(min(qw0 + 32, a.S), L);
  const int nt = (kend + BT - 1) / BT;

  const i32x4_t rk = buffer_rsrc(K + rowb * a.ldk + (int64_t)kvh * HD);
  const i32x4_t rv = buffer_rsrc(V + rowb * a.ldv + (int64_t)kvh * HD);
  TileDma<HD, FW_NT> dkm, dvm;
  dkm.init(lane, a.ldk);
  dvm.init(lane, a.ldv);
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(smem);  // [FW_NST][K | V]
  // K/V tile t goes to stage t % FW_NST, FW_NST - 1 tiles ahead of its use
  for (int p = 0; p < FW_NST - 1 && p < nt; ++p) {
    dkm.issue(lds0 + p * 2 * TB, wave, p * BT, kend, rk);
    dvm.issue(lds0 + p * 2 * TB + TB, wave, p * BT, kend, rv);
  }
  int rd = 0, wr = FW_NST - 1;
  for (int t = 0; t < nt; ++t) {
    const int k0 = t * BT;
    wait_tiles<2 * TileDma<HD, FW_NT>::ITEMS>(min(FW_NST - 2, nt - 1 - t));
    __syncthreads();  // tile t everywhere; stage wr (tile t - 1) is no longer read
    if (t + FW_NST - 1 < nt) {
      dkm.issue(lds0 + wr * 2 * TB, wave, (t + FW_NST - 1) * BT, kend, rk);
      dvm.issue(lds0 + wr * 2 * TB + TB, wave, (t + FW_NST - 1) * BT, kend, rv);
    }
    const bf16_t* kt = reinterpret_cast<const bf16_t*>(smem + rd * 2 * TB);
    rd = rd + 1 == FW_NST ? 0 : rd + 1;
    wr = wr + 1 == FW_NST ? 0 : wr + 1;
    if (k0 >= kend_w) continue;
    const bf16_t* vt = kt + BT * HD;
    const bool masked = k0 + BT - 1 > qw0 || k0 + BT > kend;
    bf16x8_t dsk[2][2];
    // K / V fragments of the next (block, k-step) are read while the
    // current step's four independent MFMAs run
    bf16x8_t ka[2], va[2];
    ka[0] = frag_row<HD>(kt, c, g);
    va[0] = frag_row<HD>(vt, c, g);
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      f32x4_t st[2], dpt[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        st[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        dpt[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int kk = 0; kk < HD / 32; ++kk) {
        const int i = blk * (HD / 32) + kk, cur = i & 1;
        if (i + 1 < 4 * (HD / 32)) {
          const int nb = (i + 1) / (HD / 32), nk = (i + 1) % (HD / 32);
          ka[cur ^ 1] = frag_row<HD>(kt, nb * 16 + c, g + 4 * nk);
          va[cur ^ 1] = frag_row<HD>(vt, nb * 16 + c, g + 4 * nk);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          st[j] = mfma16(ka[cur], qf[j][kk], st[j]);
          dpt[j] = mfma16(va[cur], df[j][kk], dpt[j]);
        }
      }
      // the mask as one uniform branch over the block's eight scores (most
      // tiles skip it), not a select per score
      float x[2][4];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) x[j][r] = st[j][r] * cs - l2[j];
      if (masked) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = k0 + blk * 16 + 4 * g + r;
            x[j][r] = (key <= qi[j] && key < kend) ? x[j][r] : -INFINITY;
          }
      }
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(x[j][r]);
          dsk[j][blk >> 1][(blk & 1) * 4 + r] = (__bf16)(p * (dpt[j][r] - dl[j]));
        }
    }
    // K^T fragments of the dQ update: a ring of KA reads in flight
    constexpr int NC = 2 * (HD / 16), KA = 4;
    bf16x8_t kc[KA];
#pragma unroll
    for (int i = 0; i < KA; ++i) kc[i] = frag_col<HD>(kt, 32 * (i & 1), g, 16 * (i >> 1), c);
#pragma unroll
    for (int i = 0; i < NC; ++i) {  // i = 2 db + kk
      const int db = i >> 1, kk = i & 1, cur = i % KA;
      __builtin_amdgcn_sched_barrier(0);
      dq[0][db] = mfma16(dsk[0][kk], kc[cur], dq[0][db]);
      dq[1][db] = mfma16(dsk[1][kk], kc[cur], dq[1][db]);
      if (i + KA < NC) kc[cur] = frag_col<HD>(kt, 32 * ((i + KA) & 1), g, 16 * ((i + KA) >> 1), c);
    }
  }
  dma_wait();
  bf16_t* DQ = reinterpret_cast<bf16_t*>(a.dq);
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int q = qw0 + j * 16 + 4 * g + r;
      if (q < a.S) {
        if (a.rope) rope_back<HD>(dq[j], r, a.pos, rowb + q, a.rope, a.max_pos, c);
#pragma unroll
        for (int db = 0; db < HD / 16; ++db)
          DQ[(rowb + q) * a.lddq + (int64_t)h * HD + db * 16 + c] = f32_to_bf16(dq[j][db][r] * a.scale);
      }
    }
}

// ------------------------------------------------------------------ launch
template <typename Kern>
static hipError_t set_lds(Kern kern, size_t bytes) {
  return hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

template <int HD, int HPW>
static hipError_t fwd_hpw(const AttnDesc& a, hipStream_t s) {
  const size_t lds = (size_t)FW_NST * 2 * BT * HD * sizeof(bf16_t);  // stages x (K + V)
  static bool once = false;
  if (!once) {
    hipError_t e = set_lds(attn_fwd_mfma<HD, HPW>, lds);
    if (e != hipSuccess) return e;
    once = true;
  }
  constexpr int QB = (FW_WAVES / HPW) * 32;
  dim3 grid((a.S + QB - 1) / QB, a.Hq / HPW, a.B);
  hipLaunchKernelGGL((attn_fwd_mfma<HD, HPW>), grid, dim3(FW_NT), lds, s, a);
  return hipGetLastError();
}

template <int HD>
static hipError_t fwd(const AttnDesc& a, hipStream_t s) {
  const int grp = a.Hq / a.Hkv;
  if (grp % 4 == 0) return fwd_hpw<HD, 4>(a, s);
  if (grp % 2 == 0) return fwd_hpw<HD, 2>(a, s);
  return fwd_hpw<HD, 1>(a, s);
}

template <int HD, int HPW>
static hipError_t dq_hpw(const AttnDesc& a, hipStream_t s) {
  const size_t lds = (size_t)FW_NST * 2 * BT * HD * sizeof(bf16_t);  // stages x (K + V)
  static bool once = false;
  if (!once) {
    hipError_t e = set_lds(attn_dq_mfma<HD, HPW>, lds);
    if (e != hipSuccess) return e;
    once = true;
  }
  constexpr int QB = (FW_WAVES / HPW) * 32;
  dim3 grid((a.S + QB - 1) / QB, a.Hq / HPW, a.B);
  hipLaunchKernelGGL((attn_dq_mfma<HD, HPW>), grid, dim3(FW_NT), lds, s, a);
  return hipGetLastError();
}

template <int HD>
static hipError_t bwd(const AttnDesc& a, hipStream_t s) {
  const size_t lds_kv = dkv_lds_bytes<HD>();
  static bool once = false;
  if (!once) {
    hipError_t e = set_lds(attn_dkv_mfma<HD>, lds_kv);
    if (e != hipSuccess) return e;
    once = true;
  }
  const int64_t rows = (int64_t)a.B * a.Hq * a.S;
  if (!a.delta_ready) {
    hipLaunchKernelGGL(attn_delta_mfma<HD>, dim3((unsigned)((rows * 64 + 255) / 256)), dim3(256), 0,
                       s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 gk((a.S + KV_KB - 1) / KV_KB, a.Hkv, a.B);
  hipLaunchKernelGGL(attn_dkv_mfma<HD>, gk, dim3(KV_NT), lds_kv, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int grp = a.Hq / a.Hkv;
  if (grp % 4 == 0) return dq_hpw<HD, 4>(a, s);
  if (grp % 2 == 0) return dq_hpw<HD, 2>(a, s);
  return dq_hpw<HD, 1>(a, s);
}

static bool mfma_ok(const AttnDesc& a) {
  if (a.hd != 64 && a.hd != 128) return false;
  // 16-byte aligned rows and column offsets for the vector loads
  const int64_t lds[] = {a.ldq, a.ldk, a.ldv, a.ldo};
  for (int64_t l : lds)
    if (l % 8) return false;
  const uintptr_t p = (uintptr_t)a.q | (uintptr_t)a.k | (uintptr_t)a.v | (uintptr_t)a.o;
  // K/V tiles are copied with 32-bit byte offsets from the batch row origin
  const int64_t lim = (int64_t)1 << 31;
  if (((int64_t)a.S + BT) * a.ldk * 2 >= lim || ((int64_t)a.S + BT) * a.ldv * 2 >= lim) return false;
  return p % 16 == 0;
}

hipError_t launch_attn_fwd_mfma(const AttnDesc& a, hipStream_t s, bool* handled) {
  *handled = mfma_ok(a);
  if (!*handled) return hipSuccess;
  return a.hd == 128 ? fwd<128>(a, s) : fwd<64>(a, s);
}

// dq / dk leave with the inverse RoPE applied when a.rope is set.
hipError_t launch_attn_bwd_mfma(const AttnDesc& a, hipStream_t s, bool* handled) {
  *handled = mfma_ok(a) && a.lddo % 8 == 0 && (uintptr_t)a.dout % 16 == 0;
  if (!*handled) return hipSuccess;
  return a.hd == 128 ? bwd<128>(a, s) : bwd<64>(a, s);
}

}  // namespace zl
