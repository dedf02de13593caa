// MFMA flash attention for bf16, head_dim 64 or 128 (the decoder layers of
// f_k in Eq. (1)): causal, GQA (q-head h reads kv-head h / (Hq / Hkv)),
// right padding by seq_len, scores q.k / sqrt(hd), fp32 softmax statistics.
//
// MFMA 16x16x32 bf16.  Lane l of a wave: c = l % 16 (output column), g = l / 16.
//  - Forward: each wave owns 16 queries.  S^T = K Q^T puts the scores of one
//    query in one lane column (keys 16*blk + 4g + r), so the online softmax
//    statistics live per lane and P feeds O^T += V^T P^T straight from
//    registers: the MFMA only needs A and B to agree on which 8 keys each lane
//    group carries, {32kk + 4g + r} and {32kk + 16 + 4g + r}.  V is staged in
//    LDS transposed ([dim][key]).
//  - dK/dV: one workgroup per (key block of 64, kv-head); it walks every
//    q-head of its group and every later query tile, so the GQA sum needs no
//    cross-workgroup reduction.  S = Q K^T keeps one key per lane column.
//  - dQ: one workgroup per (query block of 64, q-head), as the forward.
// LDS rows are XOR-swizzled in 16-byte chunks against bank conflicts.
#include "common.h"

namespace zl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

namespace {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int BT = 64;  // rows per tile (queries or keys)

__device__ inline f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int HD>
__device__ inline int swz_nat(int row) {
  return HD == 128 ? (row & 15) : ((row >> 1) & 7);
}
__device__ inline int swz_tr(int row) { return (row >> 1) & 7; }

__device__ inline bf16x8_t zero8() {
  bf16x8_t z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.f;
  return z;
}

__device__ inline bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

__device__ inline __bf16 to_bf16(float f) {
  return __builtin_bit_cast(__bf16, f32_to_bf16(f));
}

// Transpose an 8x8 bf16 block held as 8 rows (uint4 = 8 bf16 each).
__device__ inline void tr8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
  const uint32_t* iw = reinterpret_cast<const uint32_t*>(in);
  uint32_t* ow = reinterpret_cast<uint32_t*>(out);
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = iw[(2 * q) * 4 + j / 2];
      const uint32_t hi = iw[(2 * q + 1) * 4 + j / 2];
      ow[j * 4 + q] = __builtin_amdgcn_perm(hi, lo, (j & 1) ? 0x07060302u : 0x05040100u);
    }
}

// Natural tile: lds[i][0..HD) = G[rowbase + row0 + i][col0 ..], rows >= nvalid zero.
template <int HD>
__device__ inline void load_nat(bf16_t* lds, const bf16_t* G, int64_t ld, int64_t rowbase,
                                int row0, int nvalid, int64_t col0) {
  constexpr int CH = HD / 8;
  for (int c = threadIdx.x; c < BT * CH; c += 256) {
    const int i = c / CH, ch = c % CH;
    const int t = row0 + i;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t < nvalid) v = *reinterpret_cast<const uint4*>(G + (rowbase + t) * ld + col0 + ch * 8);
    *reinterpret_cast<uint4*>(lds + i * HD + ((ch ^ swz_nat<HD>(i)) * 8)) = v;
  }
}

// Transposed tile: lds[d][i] = G[rowbase + row0 + i][col0 + d], 64 columns i.
template <int HD>
__device__ inline void load_tr(bf16_t* lds, const bf16_t* G, int64_t ld, int64_t rowbase,
                               int row0, int nvalid, int64_t col0) {
  for (int bi = threadIdx.x; bi < 8 * (HD / 8); bi += 256) {
    const int kb = bi & 7, db = bi >> 3;
    uint4 in[8], out[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int r = row0 + kb * 8 + t;
      in[t] = r < nvalid ? *reinterpret_cast<const uint4*>(G + (rowbase + r) * ld + col0 + db * 8)
                         : make_uint4(0, 0, 0, 0);
    }
    tr8x8(in, out);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int d = db * 8 + j;
      *reinterpret_cast<uint4*>(lds + d * BT + ((kb ^ swz_tr(d)) * 8)) = out[j];
    }
  }
}

// 16-byte fragment of a natural tile: row i, 16-byte chunk ch.
template <int HD>
__device__ inline bf16x8_t frag_nat(const bf16_t* lds, int i, int ch) {
  return *reinterpret_cast<const bf16x8_t*>(lds + i * HD + ((ch ^ swz_nat<HD>(i)) * 8));
}

// Fragment of a transposed tile for lane group g and key/query step kk:
// columns {32kk + 4g .. +3} then {32kk + 16 + 4g .. +3} of row d.
__device__ inline bf16x8_t frag_tr(const bf16_t* lds, int d, int kk, int g) {
  const int k1 = 32 * kk + 4 * g, k2 = k1 + 16;
  const bf16_t* row = lds + d * BT;
  const uint2 a = *reinterpret_cast<const uint2*>(row + (((k1 >> 3) ^ swz_tr(d)) * 8) + ((k1 >> 2) & 1) * 4);
  const uint2 b = *reinterpret_cast<const uint2*>(row + (((k2 >> 3) ^ swz_tr(d)) * 8) + ((k2 >> 2) & 1) * 4);
  return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// Inverse (transposed) rotate-half RoPE of one row held as HD/16 register
// blocks x[db][r] (dims 16*db + c16): pairs (j, j + HD/2) sit HD/32 blocks
// apart in the same lane.  du_j = du'_j c + du'_{j+h} s,
// du_{j+h} = du'_{j+h} c - du'_j s.
template <int HD>
__device__ inline void rope_back(f32x4_t (&x)[HD / 16], int r, const int32_t* pos, int64_t row,
                                 const float2* table, int max_pos, int c16) {
  int p = pos[row];
  p = p < 0 ? 0 : (p >= max_pos ? max_pos - 1 : p);
  constexpr int HB = HD / 32;
#pragma unroll
  for (int db = 0; db < HB; ++db) {
    const float2 cs = table[(int64_t)p * (HD / 2) + db * 16 + c16];
    const float a = x[db][r], b = x[db + HB][r];
    x[db][r] = a * cs.x + b * cs.y;
    x[db + HB][r] = b * cs.x - a * cs.y;
  }
}

}  // namespace

// ------------------------------------------------------------------ forward
template <int HD>
__global__ void __launch_bounds__(256) attn_fwd_mfma(AttnDesc a) {
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Vt = Ks + BT * HD;
  const int qb = gridDim.x - 1 - blockIdx.x;  // longest causal rows first
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h / (a.Hq / a.Hkv);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c16 = lane & 15, g = lane >> 4;
  const int L = a.seq_lens[b];
  const int q0 = qb * BT;
  const int qi = q0 + wave * 16 + c16;
  const int64_t rowb = (int64_t)b * a.S;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q);
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k);
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v);

  bf16x8_t qf[HD / 32];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk)
    qf[kk] = qi < a.S ? *reinterpret_cast<const bf16x8_t*>(Q + (rowb + qi) * a.ldq +
                                                           (int64_t)h * HD + 8 * g + 32 * kk)
                      : zero8();
  f32x4_t o[HD / 16];
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, lsum = 0.f;
  const float cs = a.scale * LOG2E;
  const int kend = min(min(q0 + BT, a.S), L);

  for (int k0 = 0; k0 < kend; k0 += BT) {
    __syncthreads();
    load_nat<HD>(Ks, K, a.ldk, rowb, k0, kend, (int64_t)kvh * HD);
    load_tr<HD>(Vt, V, a.ldv, rowb, k0, kend, (int64_t)kvh * HD);
    __syncthreads();
    f32x4_t s[4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      s[blk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < HD / 32; ++kk)
        s[blk] = mfma16(frag_nat<HD>(Ks, blk * 16 + c16, g + 4 * kk), qf[kk], s[blk]);
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 4; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + blk * 16 + 4 * g + r;
        const bool ok = key < kend && key <= qi;
        const float v = ok ? s[blk][r] * cs : -INFINITY;
        s[blk][r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(m, tmax);
    const float alpha = mnew == -INFINITY ? 1.f : exp2f(m - mnew);
    float psum = 0.f;
    bf16x8_t pf[2];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = s[blk][r] == -INFINITY ? 0.f : exp2f(s[blk][r] - mnew);
        psum += p;
        pf[blk >> 1][(blk & 1) * 4 + r] = to_bf16(p);
      }
    lsum = lsum * alpha + psum;
    m = mnew;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) {
      o[db] *= alpha;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) o[db] = mfma16(frag_tr(Vt, db * 16 + c16, kk, g), pf[kk], o[db]);
    }
  }
  lsum += __shfl_xor(lsum, 16, 64);
  lsum += __shfl_xor(lsum, 32, 64);
  if (qi < a.S) {
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    bf16_t* O = reinterpret_cast<bf16_t*>(a.o) + (rowb + qi) * a.ldo + (int64_t)h * HD;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) {
      ushort4 w = make_ushort4(f32_to_bf16(o[db][0] * inv), f32_to_bf16(o[db][1] * inv),
                               f32_to_bf16(o[db][2] * inv), f32_to_bf16(o[db][3] * inv));
      *reinterpret_cast<ushort4*>(O + db * 16 + 4 * g) = w;
    }
    if (g == 0)
      a.lse[((int64_t)b * a.Hq + h) * a.S + qi] = lsum > 0.f ? m * LN2 + __logf(lsum) : -INFINITY;
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
template <int HD>
__global__ void __launch_bounds__(256) attn_dkv_mfma(AttnDesc a) {
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* Qs = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Qt = Qs + BT * HD;
  bf16_t* Ds = Qt + BT * HD;
  bf16_t* Dt = Ds + BT * HD;
  float* lse2s = reinterpret_cast<float*>(Dt + BT * HD);
  float* dels = lse2s + BT;
  const int kblk = gridDim.x - 1 - blockIdx.x;  // keys with the most queries first
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int grp = a.Hq / a.Hkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c16 = lane & 15, g = lane >> 4;
  const int L = a.seq_lens[b];
  const int k0 = kblk * BT;
  const int kj = k0 + wave * 16 + c16;  // this lane's key
  const int klim = min(a.S, L);
  const int64_t rowb = (int64_t)b * a.S;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q);
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k);
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v);
  const bf16_t* DO = reinterpret_cast<const bf16_t*>(a.dout);

  bf16x8_t kf[HD / 32], vf[HD / 32];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk) {
    const int64_t off = 8 * g + 32 * kk;
    kf[kk] = kj < klim ? *reinterpret_cast<const bf16x8_t*>(K + (rowb + kj) * a.ldk + (int64_t)kvh * HD + off)
                       : zero8();
    vf[kk] = kj < klim ? *reinterpret_cast<const bf16x8_t*>(V + (rowb + kj) * a.ldv + (int64_t)kvh * HD + off)
                       : zero8();
  }
  f32x4_t dk[HD / 16], dv[HD / 16];
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) {
    dk[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    dv[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const float cs = a.scale * LOG2E;
  if (k0 < klim) {
    for (int hh = 0; hh < grp; ++hh) {
      const int h = kvh * grp + hh;
      const float* lse = a.lse + ((int64_t)b * a.Hq + h) * a.S;
      const float* del = a.delta + ((int64_t)b * a.Hq + h) * a.S;
      for (int q0 = k0; q0 < a.S; q0 += BT) {
        __syncthreads();
        load_nat<HD>(Qs, Q, a.ldq, rowb, q0, a.S, (int64_t)h * HD);
        load_tr<HD>(Qt, Q, a.ldq, rowb, q0, a.S, (int64_t)h * HD);
        load_nat<HD>(Ds, DO, a.lddo, rowb, q0, a.S, (int64_t)h * HD);
        load_tr<HD>(Dt, DO, a.lddo, rowb, q0, a.S, (int64_t)h * HD);
        if (threadIdx.x < BT) {
          const int q = q0 + threadIdx.x;
          lse2s[threadIdx.x] = q < a.S ? lse[q] * LOG2E : -INFINITY;
          dels[threadIdx.x] = q < a.S ? del[q] : 0.f;
        }
        __syncthreads();
        bf16x8_t pk[2], dsk[2];
#pragma unroll
        for (int qb = 0; qb < 4; ++qb) {
          f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < HD / 32; ++kk) {
            s = mfma16(frag_nat<HD>(Qs, qb * 16 + c16, g + 4 * kk), kf[kk], s);
            dp = mfma16(frag_nat<HD>(Ds, qb * 16 + c16, g + 4 * kk), vf[kk], dp);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ql = qb * 16 + 4 * g + r;
            const int q = q0 + ql;
            const float l2 = lse2s[ql];
            const bool ok = q < a.S && kj <= q && kj < klim && l2 != -INFINITY;
            const float p = ok ? exp2f(s[r] * cs - l2) : 0.f;
            const float ds = p * (dp[r] - dels[ql]);
            pk[qb >> 1][(qb & 1) * 4 + r] = to_bf16(p);
            dsk[qb >> 1][(qb & 1) * 4 + r] = to_bf16(ds);
          }
        }
#pragma unroll
        for (int db = 0; db < HD / 16; ++db)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            dv[db] = mfma16(pk[kk], frag_tr(Dt, db * 16 + c16, kk, g), dv[db]);
            dk[db] = mfma16(dsk[kk], frag_tr(Qt, db * 16 + c16, kk, g), dk[db]);
          }
      }
    }
  }
  bf16_t* DK = reinterpret_cast<bf16_t*>(a.dk);
  bf16_t* DV = reinterpret_cast<bf16_t*>(a.dv);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int key = k0 + wave * 16 + 4 * g + r;
    if (key < a.S) {
      if (a.rope) rope_back<HD>(dk, r, a.pos, rowb + key, a.rope, a.max_pos, c16);
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        const int64_t col = (int64_t)kvh * HD + db * 16 + c16;
        DK[(rowb + key) * a.lddk + col] = f32_to_bf16(dk[db][r] * a.scale);
        DV[(rowb + key) * a.lddv + col] = f32_to_bf16(dv[db][r]);
      }
    }
  }
}

// ----------------------------------------------------------------------- dQ
template <int HD>
__global__ void __launch_bounds__(256) attn_dq_mfma(AttnDesc a) {
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Kt = Ks + BT * HD;
  bf16_t* Vs = Kt + BT * HD;
  const int qblk = gridDim.x - 1 - blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h / (a.Hq / a.Hkv);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c16 = lane & 15, g = lane >> 4;
  const int L = a.seq_lens[b];
  const int q0 = qblk * BT;
  const int qi = q0 + wave * 16 + c16;
  const int64_t rowb = (int64_t)b * a.S;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q);
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k);
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v);
  const bf16_t* DO = reinterpret_cast<const bf16_t*>(a.dout);

  bf16x8_t qf[HD / 32], df[HD / 32];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk) {
    const int64_t col = (int64_t)h * HD + 8 * g + 32 * kk;
    qf[kk] = qi < a.S ? *reinterpret_cast<const bf16x8_t*>(Q + (rowb + qi) * a.ldq + col) : zero8();
    df[kk] = qi < a.S ? *reinterpret_cast<const bf16x8_t*>(DO + (rowb + qi) * a.lddo + col) : zero8();
  }
  const float l2 = qi < a.S ? a.lse[((int64_t)b * a.Hq + h) * a.S + qi] * LOG2E : -INFINITY;
  const float dl = qi < a.S ? a.delta[((int64_t)b * a.Hq + h) * a.S + qi] : 0.f;
  f32x4_t dq[HD / 16];
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) dq[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const float cs = a.scale * LOG2E;
  const int kend = min(min(q0 + BT, a.S), L);

  for (int k0 = 0; k0 < kend; k0 += BT) {
    __syncthreads();
    load_nat<HD>(Ks, K, a.ldk, rowb, k0, kend, (int64_t)kvh * HD);
    load_tr<HD>(Kt, K, a.ldk, rowb, k0, kend, (int64_t)kvh * HD);
    load_nat<HD>(Vs, V, a.ldv, rowb, k0, kend, (int64_t)kvh * HD);
    __syncthreads();
    bf16x8_t dsk[2];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      f32x4_t st = f32x4_t{0.f, 0.f, 0.f, 0.f}, dpt = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < HD / 32; ++kk) {
        st = mfma16(frag_nat<HD>(Ks, blk * 16 + c16, g + 4 * kk), qf[kk], st);
        dpt = mfma16(frag_nat<HD>(Vs, blk * 16 + c16, g + 4 * kk), df[kk], dpt);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + blk * 16 + 4 * g + r;
        const bool ok = key < kend && key <= qi && l2 != -INFINITY;
        const float p = ok ? exp2f(st[r] * cs - l2) : 0.f;
        dsk[blk >> 1][(blk & 1) * 4 + r] = to_bf16(p * (dpt[r] - dl));
      }
    }
#pragma unroll
    for (int db = 0; db < HD / 16; ++db)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) dq[db] = mfma16(dsk[kk], frag_tr(Kt, db * 16 + c16, kk, g), dq[db]);
  }
  bf16_t* DQ = reinterpret_cast<bf16_t*>(a.dq);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int q = q0 + wave * 16 + 4 * g + r;
    if (q < a.S) {
      if (a.rope) rope_back<HD>(dq, r, a.pos, rowb + q, a.rope, a.max_pos, c16);
#pragma unroll
      for (int db = 0; db < HD / 16; ++db)
        DQ[(rowb + q) * a.lddq + (int64_t)h * HD + db * 16 + c16] = f32_to_bf16(dq[db][r] * a.scale);
    }
  }
}

// ------------------------------------------------------------------ launch
template <typename K>
static hipError_t set_lds(K kern, size_t bytes) {
  return hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

template <int HD>
static hipError_t fwd(const AttnDesc& a, hipStream_t s) {
  const size_t lds = (size_t)2 * BT * HD * sizeof(bf16_t);
  static bool once = false;
  if (!once) {
    hipError_t e = set_lds(attn_fwd_mfma<HD>, lds);
    if (e != hipSuccess) return e;
    once = true;
  }
  dim3 grid((a.S + BT - 1) / BT, a.Hq, a.B);
  hipLaunchKernelGGL(attn_fwd_mfma<HD>, grid, dim3(256), lds, s, a);
  return hipGetLastError();
}

template <int HD>
static hipError_t bwd(const AttnDesc& a, hipStream_t s) {
  const size_t lds_kv = (size_t)4 * BT * HD * sizeof(bf16_t) + 2 * BT * sizeof(float);
  const size_t lds_q = (size_t)3 * BT * HD * sizeof(bf16_t);
  static bool once = false;
  if (!once) {
    hipError_t e = set_lds(attn_dkv_mfma<HD>, lds_kv);
    if (e == hipSuccess) e = set_lds(attn_dq_mfma<HD>, lds_q);
    if (e != hipSuccess) return e;
    once = true;
  }
  const int64_t rows = (int64_t)a.B * a.Hq * a.S;
  hipLaunchKernelGGL(attn_delta_mfma<HD>, dim3((unsigned)((rows * 64 + 255) / 256)), dim3(256), 0,
                     s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 gk((a.S + BT - 1) / BT, a.Hkv, a.B);
  hipLaunchKernelGGL(attn_dkv_mfma<HD>, gk, dim3(256), lds_kv, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 gq((a.S + BT - 1) / BT, a.Hq, a.B);
  hipLaunchKernelGGL(attn_dq_mfma<HD>, gq, dim3(256), lds_q, s, a);
  return hipGetLastError();
}

static bool mfma_ok(const AttnDesc& a) {
  if (a.hd != 64 && a.hd != 128) return false;
  // 16-byte aligned rows and column offsets for the vector loads
  const int64_t lds[] = {a.ldq, a.ldk, a.ldv, a.ldo};
  for (int64_t l : lds)
    if (l % 8) return false;
  const uintptr_t p = (uintptr_t)a.q | (uintptr_t)a.k | (uintptr_t)a.v | (uintptr_t)a.o;
  return p % 16 == 0;
}

hipError_t launch_attn_fwd_mfma(const AttnDesc& a, hipStream_t s, bool* handled) {
  *handled = mfma_ok(a);
  if (!*handled) return hipSuccess;
  return a.hd == 128 ? fwd<128>(a, s) : fwd<64>(a, s);
}

hipError_t launch_attn_bwd_mfma(const AttnDesc& a, hipStream_t s, bool* handled) {
  // dq / dk leave with the inverse RoPE applied when a.rope is set
  *handled = mfma_ok(a) && a.lddo % 8 == 0 && (uintptr_t)a.dout % 16 == 0;
  if (!*handled) return hipSuccess;
  return a.hd == 128 ? bwd<128>(a, s) : bwd<64>(a, s);
}

}  // namespace zl
