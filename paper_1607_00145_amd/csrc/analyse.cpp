// analyse.cpp -- descriptor analyser: the host-side stand-in for the paper's
// code generator (Sec. 3.2-3.3, Sec. 6).  Runs once per contraction shape and
// makes no HIP call.
//
//   1. parse and validate the three mode lists (Sec. 2.2, footnote 9);
//   2. classify indices into I_m, I_n, I_k (Listing 5: I_m = A ∩ C,
//      I_n = B ∩ C, I_k = A ∩ B);
//   3. drop extent-1 indices and merge indices of one set that are adjacent
//      in memory in every tensor holding them into super-indices (Sec. 6,
//      footnote 18, applied to strides so that it also covers non-dense
//      views);
//   4. choose the row and column operands of the macro-kernel: C's
//      stride-one index goes to the column side, where the kernel stores C
//      contiguously (the operand exchange of Listing 7, mirrored for the
//      MFMA result layout);
//   5. order every set so each operand's stride-one index leads where
//      possible (Sec. 3.2.1: keep the stride-one index inside the packed
//      sub-tensor);
//   6. choose the tile shape and the K box -- a sub-tensor of fixed shape
//      over the contracted indices, splitting one index into blocks
//      (Sec. 3.2.1, Examples 1-2: index reinterpretation) -- and the gather
//      mode of each operand.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cctype>
#include <new>
#include <sstream>

#include "plan.hpp"
#include "tiles.hpp"

namespace gett {
namespace {

gett_status_t parse_modes(const char *s, std::vector<std::string> &out)
{
    out.clear();
    if (!s) return GETT_ERROR_INVALID_VALUE;
    if (!strchr(s, ',')) {
        for (const char *p = s; *p; ++p)
            if (*p != ' ') out.push_back(std::string(1, *p));
        return GETT_SUCCESS;
    }
    std::string cur;
    for (const char *p = s;; ++p) {
        if (*p == ',' || *p == 0) {
            if (cur.empty()) {
                if (*p == 0 && !out.empty()) break;   // one trailing comma
                return GETT_ERROR_INVALID_INDICES;
            }
            out.push_back(cur);
            cur.clear();
            if (*p == 0) break;
        } else if (*p != ' ') {
            cur.push_back(*p);
        }
    }
    return GETT_SUCCESS;
}

struct Tensor {
    std::vector<std::string> modes;
    std::vector<int64_t> ext, str;
    int find(const std::string &n) const
    {
        for (size_t i = 0; i < modes.size(); ++i)
            if (modes[i] == n) return (int)i;
        return -1;
    }
};

gett_status_t load_tensor(const char *m, const int64_t *e, const int64_t *s, Tensor &t)
{
    gett_status_t st = parse_modes(m, t.modes);
    if (st != GETT_SUCCESS) return st;
    const size_t n = t.modes.size();
    if (n > GETT_MAX_RANK) return GETT_ERROR_NOT_SUPPORTED;
    if (n && !e) return GETT_ERROR_INVALID_VALUE;
    for (size_t i = 0; i < n; ++i)
        for (size_t j = i + 1; j < n; ++j)
            if (t.modes[i] == t.modes[j]) return GETT_ERROR_INVALID_INDICES;
    t.ext.assign(e, e + n);
    for (int64_t v : t.ext)
        if (v < 0 || v > INT32_MAX) return GETT_ERROR_INVALID_VALUE;
    if (s) {
        t.str.assign(s, s + n);
    } else {   // Fortran layout: the first index is stride-one (Sec. 2.2)
        t.str.resize(n);
        int64_t acc = 1;
        for (size_t i = 0; i < n; ++i) {
            t.str[i] = acc;
            acc *= std::max<int64_t>(t.ext[i], 1);
        }
    }
    for (size_t i = 0; i < n; ++i) {
        if (t.str[i] < 0) return GETT_ERROR_INVALID_VALUE;
        if (t.ext[i] > 1 && t.str[i] < 1) return GETT_ERROR_INVALID_VALUE;
    }
    return GETT_SUCCESS;
}

// Largest element offset of a tensor (INT64_MAX beyond 2^62).
int64_t max_offset(const Tensor &t)
{
    const int64_t cap = (int64_t)1 << 62;
    int64_t m = 0;
    for (size_t i = 0; i < t.modes.size(); ++i) {
        if (t.ext[i] <= 1) continue;
        if (t.str[i] >= cap || (t.ext[i] - 1) > cap / t.str[i]) return INT64_MAX;
        m += (t.ext[i] - 1) * t.str[i];
        if (m >= cap) return INT64_MAX;
    }
    return m;
}

}  // namespace

// Strides that may send two elements to one address are refused: sorted by
// stride, each index must step over the whole span of the previous ones.
bool strides_injective(int n, const int64_t *ext, const int64_t *str)
{
    std::vector<std::pair<int64_t, int64_t>> v;   // (stride, extent)
    for (int i = 0; i < n; ++i)
        if (ext[i] > 1) v.push_back({str[i], ext[i]});
    std::sort(v.begin(), v.end());
    int64_t span = 1;   // one past the largest offset reachable so far
    for (auto &p : v) {
        if (p.first < span) return false;
        span = p.first * (p.second - 1) + span;
    }
    return true;
}

namespace {

bool c_is_injective(const Tensor &c)
{
    return strides_injective((int)c.modes.size(), c.ext.data(), c.str.data());
}

// Merge p then q (p fastest) when q follows p in memory in every tensor that
// holds them (Sec. 6, footnote 18).
void merge_set(std::vector<Index> &set, bool useA, bool useB, bool useC,
               std::vector<std::string> &log)
{
    bool changed = true;
    while (changed) {
        changed = false;
        for (size_t p = 0; p < set.size() && !changed; ++p)
            for (size_t q = 0; q < set.size() && !changed; ++q) {
                if (p == q) continue;
                const Index &P = set[p], &Q = set[q];
                auto follows = [&](int64_t sp, int64_t sq) { return sq == sp * P.extent; };
                if (useA && !follows(P.strA, Q.strA)) continue;
                if (useB && !follows(P.strB, Q.strB)) continue;
                if (useC && !follows(P.strC, Q.strC)) continue;
                Index M = P;
                M.name = "(" + P.name + "," + Q.name + ")";
                M.extent = P.extent * Q.extent;
                log.push_back(M.name);
                set[p] = M;
                set.erase(set.begin() + q);
                changed = true;
            }
    }
}

const TileShape &tile_shape(gett_dtype_t dt, int t)
{
    return dt == GETT_FLOAT32 ? kTilesF32[t] : kTilesF64[t];
}
int num_tiles(gett_dtype_t dt) { return dt == GETT_FLOAT32 ? kNumTilesF32 : kNumTilesF64; }

void json_set(std::ostringstream &o, const char *key, const std::vector<Index> &set, bool A, bool B,
              bool C)
{
    o << "\"" << key << "\":[";
    for (size_t i = 0; i < set.size(); ++i) {
        const Index &x = set[i];
        o << (i ? "," : "") << "{\"name\":\"" << x.name << "\",\"extent\":" << x.extent;
        if (A) o << ",\"strideA\":" << x.strA;
        if (B) o << ",\"strideB\":" << x.strB;
        if (C) o << ",\"strideC\":" << x.strC;
        o << "}";
    }
    o << "]";
}

}  // namespace

Hooks read_hooks()
{
    Hooks h;
    const struct {
        const char *name;
        const char **slot;
    } vars[] = {{"GETT_FORCE_TILE", &h.forceTile},     {"GETT_FORCE_KIND", &h.forceKind},
                {"GETT_FORCE_KSLICES", &h.forceKslices}, {"GETT_SPLIT_F", &h.splitF},
                {"GETT_C_ORDER", &h.cOrder},           {"GETT_XCD_REMAP", &h.xcdRemap},
                {"GETT_LANE_PERM", &h.lanePerm},       {"GETT_TAIL_WGS", &h.tailWgs}};
    for (const auto &v : vars) {
        *v.slot = getenv(v.name);
        if (*v.slot) h.text += std::string(v.name) + "=" + *v.slot + ";";
    }
    // the text goes into gett_plan_describe's JSON: keep it to plain characters
    for (char &c : h.text)
        if (!(isalnum((unsigned char)c) || c == '_' || c == '=' || c == ';' || c == '-' ||
              c == '.'))
            c = '?';
    return h;
}

const char *kind_name(int k)
{
    return k == 1   ? "stream"
           : k == 2 ? "kslices"
           : k == 3 ? "tail"
           : k == 4 ? "direct"
           : k == 5 ? "direct-stream"
                    : "macro";
}

// Workgroups of a tile resident on one CU at once: the wavefronts per SIMD its
// register budget allows (a workgroup of four wavefronts puts one on each
// SIMD), within the 160 KB of LDS its packed panels take.
static double tail_occupancy(const TileShape &c, double itemB)
{
    const double lds = (double)c.nbuf * c.kt * (c.mt + c.nt + 8) * itemB;
    return std::max(1.0, std::min((double)c.wpe, std::floor(160.0 * 1024.0 / lds)));
}

// Time one CU takes, in units of one K box on a SIMD shared by two or more
// wavefronts, to run `full` workgroups of `nb` boxes and then `tail`
// workgroups of `len` boxes, `occ` of them resident at once (in that order:
// the dispatcher deals workgroups in order of their index).  The resident
// workgroups share the SIMDs evenly; a wavefront left alone on its SIMD runs
// at 0.64 of the rate of two (measured on MI355X: it waits for its own
// gathers and LDS reads).
static double cu_time(int occ, int full, double nb, int tail, double len)
{
    std::vector<double> left;
    int next = 0;
    const int n = full + tail;
    auto work = [&](int i) { return i < full ? nb : len; };
    while (next < n && (int)left.size() < occ) left.push_back(work(next++));
    double t = 0.0;
    while (!left.empty()) {
        const double w = (double)left.size();
        // (a tile that holds one wavefront per SIMD anyway has that rate in
        // its measured efficiency)
        const double rate = (left.size() >= 2 || occ < 2 ? 1.0 : 0.64) / w;   // per unit, each
        const double step = *std::min_element(left.begin(), left.end());
        t += step / rate;
        std::vector<double> still;
        for (double r : left)
            if (r - step > 1e-9) still.push_back(r - step);
        left.swap(still);
        while (next < n && (int)left.size() < occ) left.push_back(work(next++));
    }
    return t;
}

// Stream-K tail shape for T tiles of nb boxes over G tail workgroups:
// whole tiles for the complete rounds of G, the boxes of the rest in equal
// runs; every tail workgroup gets boxes.
struct TailShape {
    int64_t full = 0, wgs = 0, len = 0;
};
static TailShape tail_shape(int64_t T, int64_t nb, int64_t G)
{
    TailShape s;
    int64_t rem = T % G;
    if (rem == 0) rem = std::min<int64_t>(G, T);
    const int64_t boxes = rem * nb;
    s.len = (boxes + std::min(G, boxes) - 1) / std::min(G, boxes);
    s.full = T - rem;
    s.wgs = (boxes + s.len - 1) / s.len;
    return s;
}

namespace {

const char *mode_name(int m)
{
    return m == kGatherRowVec         ? "row-vector"
           : m == kGatherKVec         ? "k-vector"
           : m == kGatherRowVecStrided ? "row-vector-strided"
           : m == kGatherKVecStrided  ? "k-vector-strided"
                                      : "scalar";
}

}  // namespace

gett_status_t front_end(Analysis &an, gett_dtype_t dtype, const char *mC, const int64_t *eC,
                        const int64_t *sC, const char *mA, const int64_t *eA, const int64_t *sA,
                        const char *mB, const int64_t *eB, const int64_t *sB, int rank[3],
                        bool offsets31)
{
    if (dtype != GETT_FLOAT32 && dtype != GETT_FLOAT64) return GETT_ERROR_INVALID_VALUE;
    Tensor A, B, C;
    gett_status_t st;
    if ((st = load_tensor(mC, eC, sC, C)) != GETT_SUCCESS) return st;
    if ((st = load_tensor(mA, eA, sA, A)) != GETT_SUCCESS) return st;
    if ((st = load_tensor(mB, eB, sB, B)) != GETT_SUCCESS) return st;
    rank[0] = (int)C.modes.size();
    rank[1] = (int)A.modes.size();
    rank[2] = (int)B.modes.size();

    // ---- classification (Sec. 2.2; Listing 5: the three intersections) ----
    for (size_t i = 0; i < C.modes.size(); ++i) {
        const int ia = A.find(C.modes[i]), ib = B.find(C.modes[i]);
        if ((ia >= 0) == (ib >= 0)) return GETT_ERROR_INVALID_INDICES;   // in both or neither
        Index x;
        x.name = C.modes[i];
        x.extent = C.ext[i];
        x.strC = C.str[i];
        if (ia >= 0) {
            if (A.ext[ia] != C.ext[i]) return GETT_ERROR_INVALID_INDICES;
            x.strA = A.str[ia];
            an.Im.push_back(x);
        } else {
            if (B.ext[ib] != C.ext[i]) return GETT_ERROR_INVALID_INDICES;
            x.strB = B.str[ib];
            an.In.push_back(x);
        }
    }
    for (size_t i = 0; i < A.modes.size(); ++i) {
        if (C.find(A.modes[i]) >= 0) continue;
        const int ib = B.find(A.modes[i]);
        if (ib < 0) return GETT_ERROR_INVALID_INDICES;
        if (B.ext[ib] != A.ext[i]) return GETT_ERROR_INVALID_INDICES;
        Index x;
        x.name = A.modes[i];
        x.extent = A.ext[i];
        x.strA = A.str[i];
        x.strB = B.str[ib];
        an.Ik.push_back(x);
    }
    for (size_t i = 0; i < B.modes.size(); ++i)
        if (C.find(B.modes[i]) < 0 && A.find(B.modes[i]) < 0) return GETT_ERROR_INVALID_INDICES;

    an.maxOffA = max_offset(A);
    an.maxOffB = max_offset(B);
    an.maxOffC = max_offset(C);
    const int64_t lim = offsets31 ? (int64_t)INT32_MAX : INT64_MAX;
    if (an.maxOffA >= lim || an.maxOffB >= lim || an.maxOffC >= lim) return GETT_ERROR_NOT_SUPPORTED;
    if (!c_is_injective(C)) return GETT_ERROR_NOT_SUPPORTED;

    for (auto &x : an.Im) { an.sizeM *= x.extent; }
    for (auto &x : an.In) { an.sizeN *= x.extent; }
    for (auto &x : an.Ik) { an.sizeK *= x.extent; }
    an.emptyC = an.sizeM == 0 || an.sizeN == 0;
    an.emptySum = an.sizeK == 0;

    // ---- drop extent-1 indices, merge (footnote 18) ----
    auto drop1 = [](std::vector<Index> &s) {
        s.erase(std::remove_if(s.begin(), s.end(), [](const Index &x) { return x.extent == 1; }),
                s.end());
    };
    drop1(an.Im);
    drop1(an.In);
    drop1(an.Ik);
    if (!an.emptyC && !an.emptySum) {
        merge_set(an.Im, true, false, true, an.merges);
        merge_set(an.In, false, true, true, an.merges);
        merge_set(an.Ik, true, true, false, an.merges);
    }

    return GETT_SUCCESS;
}

gett_status_t analyse(gett_plan_s &plan, gett_dtype_t dtype, const char *mC, const int64_t *eC,
                      const int64_t *sC, const char *mA, const int64_t *eA, const int64_t *sA,
                      const char *mB, const int64_t *eB, const int64_t *sB, uint32_t flags,
                      const Choice *force)
{
    Analysis an;
    int rank[3];
    const gett_status_t st =
        front_end(an, dtype, mC, eC, sC, mA, eA, sA, mB, eB, sB, rank, false);
    if (st != GETT_SUCCESS) return st;

    // ---- operand roles: C's stride-one index on the column (y) side ----
    bool swap = false;
    {
        int64_t best = INT64_MAX;
        int where = 0;   // 1: I_m, 2: I_n
        for (auto &x : an.Im)
            if (x.strC < best) { best = x.strC; where = 1; }
        for (auto &x : an.In)
            if (x.strC < best) { best = x.strC; where = 2; }
        swap = where == 1 && !(flags & GETT_FLAG_NO_SWAP);
    }
    an.swapped = swap;
    std::vector<Index> Ix = swap ? an.In : an.Im;
    std::vector<Index> Iy = swap ? an.Im : an.In;
    std::vector<Index> Ik = an.Ik;
    auto sX = [swap](const Index &x) { return swap ? x.strB : x.strA; };
    auto sY = [swap](const Index &x) { return swap ? x.strA : x.strB; };

    // ---- loop orders (stride-one index first where it helps) ----
    std::stable_sort(Iy.begin(), Iy.end(), [](const Index &a, const Index &b) { return a.strC < b.strC; });
    std::stable_sort(Ix.begin(), Ix.end(), [&](const Index &a, const Index &b) { return sX(a) < sX(b); });
    {
        int64_t minX = INT64_MAX, minY = INT64_MAX;
        bool xInK = false, yInK = false;
        for (auto &x : Ix) if (sX(x) < minX) { minX = sX(x); xInK = false; }
        for (auto &x : Ik) if (sX(x) < minX) { minX = sX(x); xInK = true; }
        for (auto &x : Iy) if (sY(x) < minY) { minY = sY(x); yInK = false; }
        for (auto &x : Ik) if (sY(x) < minY) { minY = sY(x); yInK = true; }
        const bool byY = !xInK && yInK;
        std::stable_sort(Ik.begin(), Ik.end(), [&](const Index &a, const Index &b) {
            return byY ? sY(a) < sY(b) : sX(a) < sX(b);
        });
    }
    // An empty set acts as one index of extent 1 (Sec. 2.2 assumes non-empty sets).
    auto virt = [](std::vector<Index> &s) {
        if (s.empty()) {
            Index v;
            v.name = "1";
            s.push_back(v);
        }
    };
    virt(Ix);
    virt(Iy);
    virt(Ik);
    if ((int)Ix.size() > kMaxDims || (int)Iy.size() > kMaxDims || (int)Ik.size() > kMaxDims)
        return GETT_ERROR_NOT_SUPPORTED;

    // ---- K box for a given box depth: whole leading contracted indices,
    //      then a block of one index (index reinterpretation) ----
    const int VW = dtype == GETT_FLOAT32 ? 4 : 2;
    const int64_t sizeX = swap ? an.sizeN : an.sizeM;
    const int64_t sizeY = swap ? an.sizeM : an.sizeN;
    int nk = (int)Ik.size();
    // A contracted stride-one run gathered as vectors needs whole vectors per block.
    auto kvec_ok = [&](auto strOf) {
        if (strOf(Ik[0]) != 1) return false;
        if (Ik[0].extent % VW) return false;
        for (size_t i = 1; i < Ik.size(); ++i)
            if (strOf(Ik[i]) % VW) return false;
        return true;
    };
    const bool wantKvec = !(flags & GETT_FLAG_SCALAR) && (kvec_ok(sX) || kvec_ok(sY));
    int kvecIdx = 0;   // contracted index that vector gathers run along (1 after a K split)
    struct Box {
        int kj;
        int64_t tj, kbox, nblk, nsteps;
    };
    // K box of depth kt over the contracted set K (in walk order); kvi is the
    // index that contracted vector gathers run along.
    auto box_on = [&](const std::vector<Index> &K, int kvi, int kt) {
        const int nK = (int)K.size();
        Box b;
        b.kj = 0;
        int64_t prefix = 1;
        while (b.kj < nK - 1 && prefix * K[b.kj].extent <= kt) {
            prefix *= K[b.kj].extent;
            ++b.kj;
        }
        int64_t tj = std::max<int64_t>(1, std::min<int64_t>(K[b.kj].extent, kt / prefix));
        // The block of the index that vectors run along holds whole vectors.
        // A block length that divides the index (no ragged last block) is
        // preferred unless that would lose more than half of the box (92 in
        // blocks of 4 would be 23 boxes an eighth full, against 32, 32, 28).
        const bool vec = b.kj == kvi && (wantKvec || kvi > 0);
        const int64_t step = vec ? VW : 1;
        const int64_t top = vec && tj >= VW ? (tj / VW) * VW : tj;
        if (top >= step) {
            int64_t best = top;
            for (int64_t t = top; t >= step; t -= step)
                if (K[b.kj].extent % t == 0) { best = t; break; }
            tj = best * 2 > top ? best : top;
        }
        b.tj = tj;
        b.kbox = prefix * tj;
        b.nblk = (K[b.kj].extent + tj - 1) / tj;
        b.nsteps = b.nblk;
        for (int i = b.kj + 1; i < nK; ++i) b.nsteps *= K[i].extent;
        if (an.emptySum) b.nsteps = 0;
        return b;
    };
    auto box_for = [&](int kt) { return box_on(Ik, kvecIdx, kt); };

    // ---- index splitting helpers (used by the model and by the plan; see
    //      the splitting step below) ----
    auto split_front = [](std::vector<Index> &set, size_t u, size_t v, int64_t f) {
        Index in = set[u], out = set[u];
        in.extent = f;
        in.name = set[u].name + "<" + std::to_string(f);
        out.extent = set[u].extent / f;
        out.name = set[u].name + ">" + std::to_string(f);
        out.strA *= f;
        out.strB *= f;
        out.strC *= f;
        std::vector<Index> next;
        next.push_back(in);
        next.push_back(set[v]);
        if (out.extent > 1) next.push_back(out);
        for (size_t i = 0; i < set.size(); ++i)
            if (i != u && i != v) next.push_back(set[i]);
        set.swap(next);
    };
    auto pow2_part = [](int64_t e) { return e & -e; };
    auto unit_in = [](const std::vector<Index> &set, auto strOf) -> int {
        for (size_t i = 0; i < set.size(); ++i)
            if (strOf(set[i]) == 1 && set[i].extent > 1) return (int)i;
        return -1;
    };
    auto aligned = [&](const std::vector<Index> &set, auto strOf, int skip) {
        for (size_t i = 0; i < set.size(); ++i)
            if ((int)i != skip && strOf(set[i]) % VW) return false;
        return true;
    };
    const bool maySplit = !(flags & (GETT_FLAG_SCALAR | GETT_FLAG_NO_SPLIT)) && !an.emptyC &&
                          !an.emptySum;
    const int splitXK = unit_in(Ik, sX), splitYK = unit_in(Ik, sY);
    // K-box split for a box of depth kt: X's stride-one contracted index u
    // blocked by f in front of Y's stride-one contracted index v.  X runs of f
    // (a multiple of VW), at least two vectors of v per box line when the
    // box allows.  Returns f (0: no split) and the split set in `trial`.
    auto k_split = [&](int kt, std::vector<Index> &trial) -> int64_t {
        if (!maySplit || splitXK < 0 || splitYK < 0 || splitXK == splitYK ||
            Ik[splitYK].extent % VW || (int)Ik.size() >= kMaxDims)
            return 0;
        int64_t cap = 1;
        while (cap * 2 * VW <= kt) cap *= 2;
        int64_t f = std::min<int64_t>(pow2_part(Ik[splitXK].extent), cap);
        while (f > VW && f * VW * 2 > kt) f /= 2;
        trial = Ik;
        split_front(trial, (size_t)splitXK, (size_t)splitYK, f);
        if (f >= VW && kt % (f * VW) == 0 && aligned(trial, sY, 1) && aligned(Iy, sY, -1)) return f;
        return 0;
    };

    // ---- tile shape: the paper ranks candidates with a performance model
    //      (Sec. 3.4: macro-kernel time from flops / (peak * penalty), packing
    //      and unpacking time from bytes / bandwidth).  Here: MFMA time of the
    //      busiest SIMD (the tiles' wavefronts are dealt to the 1024 SIMDs of
    //      256 CUs; each wavefront's share of a tile, padding included, runs
    //      at the sustained fraction of one SIMD's peak) against the C stream
    //      through HBM at the bandwidth the tile sustains; the longer one
    //      bounds the time. ----
    const double itemB = dtype == GETT_FLOAT32 ? 4.0 : 8.0;
    const double peakSimd = (dtype == GETT_FLOAT32 ? 157.3e12 : 78.6e12) / 1024.0;
    const double bytesX = itemB * (double)sizeX * (double)an.sizeK;
    const double bytesY = itemB * (double)sizeY * (double)an.sizeK;
    const double bytesC = itemB * (double)sizeX * (double)sizeY;
    // When the row and column operands are stride-one along different
    // contracted indices, the K box is split between them (below) and both
    // are gathered in short runs whose cache lines are reused only many
    // boxes later; without a second LDS buffer the gather latency of every
    // box is exposed (measured on MI355X: 1.4-1.8x slower than the
    // double-buffered tiles of the same depth).
    // Each tile's K box is priced on the contracted order that tile gets.
    const Hooks hk = read_hooks();
    const char *ft = hk.forceTile;
    const char *fk = hk.forceKind;
    // An operand gathers in vectors when its stride-one index leads its free
    // order or the contracted order (before any index split).
    auto vecable = [&](const std::vector<Index> &I, auto strOf) {
        return strOf(I[0]) == 1 || strOf(Ik[0]) == 1;
    };
    const bool slowGather = (flags & GETT_FLAG_SCALAR) || !vecable(Ix, sX) || !vecable(Iy, sY);
    // Partial tiles (K slices, stream-K tail) are summed through the
    // workspace: the stream of partial tiles and one workgroup's reads of a
    // tile's pieces are priced at these rates (MI355X).
    constexpr double kPartialBw = 5.0e12, kSumBw = 1.0e11;
    // C's run along y: the leading y indices that follow one another in C
    int64_t cRunY = 0;
    if (!Iy.empty() && Iy[0].strC == 1) {
        cRunY = Iy[0].extent;
        for (size_t i = 1; i < Iy.size() && Iy[i].strC == cRunY; ++i) cRunY *= Iy[i].extent;
    }
    // Every (tile, kernel kind) pair is a candidate; the model ranks them.
    std::vector<Candidate> ranked;
    for (int t = 0; t < num_tiles(dtype); ++t) {
        const TileShape &c = tile_shape(dtype, t);
        const double tileBytes = (double)c.mt * c.nt * itemB;
        // a one-box tile is ranked only for a contracted set in one box whose
        // operands are both gathered in vectors: it waits for each operand's
        // gathers in turn, which element-wise gathers make long (it still
        // runs any plan it is forced onto)
        if (c.onebox && (box_for(c.kt).nsteps > 1 || slowGather) && !(ft && atoi(ft) == t) &&
            !(force && force->tile == t))
            continue;
        std::vector<Index> ksplit;
        const bool kSplitAhead = k_split(c.kt, ksplit) > 0;
        const Box b = kSplitAhead ? box_on(ksplit, 1, c.kt) : box_for(c.kt);
        const double tx = (double)((sizeX + c.mt - 1) / c.mt);
        const double ty = (double)((sizeY + c.nt - 1) / c.nt);
        // Busiest SIMD: a workgroup of four or more wavefronts is spread over
        // the four SIMDs of one CU (ceil(w / 4) on the busiest), so a CU's
        // load is counted in workgroups; smaller workgroups share SIMDs.
        const int wpt = c.wm * c.wn;
        const double waves = tx * ty * wpt;
        const double perSimd = wpt >= 4 ? std::ceil(tx * ty / 256.0) * std::ceil(wpt / 4.0)
                                        : std::ceil(waves / 1024.0);
        // The busiest CU's tiles pass through its resident slots (cu_time):
        // a last round with fewer tiles than slots leaves wavefronts alone.
        const double perSimdRun =
            wpt >= 4
                ? cu_time((int)tail_occupancy(c, itemB), (int)std::ceil(tx * ty / 256.0), 1.0, 0,
                          0.0) *
                      std::ceil(wpt / 4.0)
                : perSimd;
        const double kpad = (double)std::max<int64_t>(b.nsteps, 1) * c.kt;
        const double waveFlops = (double)(c.mt / c.wm) * (c.nt / c.wn) * kpad * 2.0;
        // A K split gathers both operands in 16-byte runs whose cache lines
        // return late: a single LDS buffer waits for them (1.4), and so does a
        // tile with one wavefront per SIMD (1.7: on the fp32 4D x 4D
        // contractions 28 and 30 of Appendix A the 128 x 128 x 32 tile took
        // 17.7 ms, the 128 x 256 x 32 tile with two wavefronts per SIMD
        // 10.5 ms).
        const double kSplitWait = !kSplitAhead || b.nsteps <= 1 ? 1.0
                                  : c.nbuf == 1                 ? 1.4
                                  : c.wpe == 1                  ? 1.7
                                                                : 1.0;
        const double tMfma = perSimdRun * waveFlops / (peakSimd * c.eff) * kSplitWait;
        // The persistent streaming kernel needs the contracted set in one box.
        const bool canStream = c.stream && b.nsteps <= 1;
        // A stream carried by fewer workgroups than CUs gets that share of the
        // bandwidth (each CU's memory pipeline has its own limit).
        const double cuShare = std::min(1.0, std::max(tx * ty, 1.0) / 256.0);
        // Latency chain: a wavefront walks its K boxes one after another and
        // waits about 1.2 us for each box's gathers when nothing else covers
        // them (measured on MI355X with one wavefront per SIMD); the busiest
        // SIMD walks perSimd wavefronts' boxes, up to four of them resident
        // and waiting together.
        auto chain = [&](double wgs, double boxes) {
            const double ps = std::max(1.0, wpt >= 4 ? std::ceil(wgs / 256.0) * std::ceil(wpt / 4.0)
                                                     : std::ceil(wgs * wpt / 1024.0));
            return ps * boxes * 1.2e-6 / std::min(ps, 4.0);
        };
        const double tChain = chain(tx * ty, (double)std::max<int64_t>(b.nsteps, 1));
        // the larger of throughput and latency bound, with near-ties broken
        // by the other (a 4-norm)
        auto bound = [](double tput, double lat) {
            const double a = tput * tput, b = lat * lat;
            return std::sqrt(std::sqrt(a * a + b * b));
        };
        for (int k = 0; k < (canStream ? 2 : 1); ++k) {
            const double bwFrac = (k ? c.sbw : c.bw) * cuShare;
            // compulsory bytes (each operand read once, C written once) plus
            // the operand panels re-read by other tiles, mostly from L2
            const double tMem = (bytesC + bytesX + bytesY +
                                 0.05 * (bytesX * (ty - 1) + bytesY * (tx - 1))) /
                                (8.0e12 * bwFrac);
            Candidate cd;
            cd.tile = t;
            cd.kind = k;
            cd.tMfma = tMfma;
            cd.tMem = tMem;
            // element-wise gathers into a single LDS buffer (the streaming
            // kernel too) wait with nothing to overlap them, as in the K split
            const double single = (slowGather && (c.nbuf == 1 || k == 1)) ? 1.4 : 1.0;
            cd.cost = bound(std::max(tMfma, tMem), tChain) * single;
            ranked.push_back(cd);
        }
        // Direct-load kernel (tiles that carry it): both operands gathered in
        // vectors.  It sustains deff of the MFMA peak where the macro-kernel
        // sustains eff; its memory stream is priced as the macro-kernel's.
        if (c.deff > 0.0f && !slowGather && !(flags & GETT_FLAG_SCALAR) && !kSplitAhead &&
            b.nsteps >= 1) {
            const double tMem = (bytesC + bytesX + bytesY +
                                 0.05 * (bytesX * (ty - 1) + bytesY * (tx - 1))) /
                                (8.0e12 * c.bw * cuShare);
            Candidate cd;
            cd.tile = t;
            cd.kind = 4;
            cd.tMfma = tMfma * c.eff / c.deff;
            cd.tMem = tMem;
            cd.cost = bound(std::max(cd.tMfma, tMem), tChain);
            ranked.push_back(cd);
        }
        // Persistent direct-load kernel (tiles that carry it): a contracted
        // set in one box, both operands gathered in vectors; its C stream is
        // priced at dsbw of the HBM peak when C's rows along y run at least a
        // tile wide, else as the macro-kernel's (short runs: measured 1-7%
        // slower than the macro-kernel on the fp64 6D contractions of
        // Appendix A whose y set leads with one index of 24, 3-5% faster
        // on those whose y set leads with a merged run of 384).
        if (c.dsbw > 0.0f && !slowGather && !(flags & GETT_FLAG_SCALAR) && !kSplitAhead &&
            b.nsteps == 1) {
            const double dbw = cRunY >= c.nt ? c.dsbw : c.bw;
            const double tMem = (bytesC + bytesX + bytesY +
                                 0.05 * (bytesX * (ty - 1) + bytesY * (tx - 1))) /
                                (8.0e12 * dbw * cuShare);
            Candidate cd;
            cd.tile = t;
            cd.kind = 5;
            cd.tMfma = tMfma;
            cd.tMem = tMem;
            cd.cost = bound(std::max(tMfma, tMem), tChain);
            ranked.push_back(cd);
        }
        // K slices: when a contracted set of many boxes meets too few tiles to
        // give every SIMD two wavefronts, P workgroups share each tile's
        // boxes.  Their partial tiles go to the workspace and the last of a
        // tile's slices to finish sums the P of them in slice order.  Priced
        // like the macro-kernel on tiles * P workgroups with ceil(boxes / P)
        // boxes each plus two boxes' worth of set-up and epilogue per
        // workgroup, plus the partial tiles' traffic, which adds to the time:
        // P tile writes and reads per tile as a stream, and the last slice's
        // P reads of one tile in turn.  Each slice keeps at least eight
        // boxes.
        if (!(flags & GETT_FLAG_WHOLE_TILES) && !an.emptyC && waves < 2048.0 &&
            b.nsteps >= 16) {
            Candidate best;
            best.tile = -1;
            for (int P = 2; P <= 256 && b.nsteps / P >= 8; P *= 2) {
                const double wgs = tx * ty * P;
                const double perSimdP =
                    wpt >= 4 ? cu_time((int)tail_occupancy(c, itemB), (int)std::ceil(wgs / 256.0),
                                       1.0, 0, 0.0) *
                                   std::ceil(wpt / 4.0)
                             : std::ceil(wgs * wpt / 1024.0);
                const double kpadP = (std::ceil((double)b.nsteps / P) + 2.0) * c.kt;
                const double tM = perSimdP * (double)(c.mt / c.wm) * (c.nt / c.wn) * kpadP * 2.0 /
                                  (peakSimd * c.eff) *
                                  (kSplitAhead && c.nbuf == 1 ? 1.4 : 1.0);
                const double shareP = std::min(1.0, wgs / 256.0);
                const double tMemP = (bytesC + bytesX + bytesY +
                                      0.05 * (bytesX * (ty - 1) + bytesY * (tx - 1))) /
                                     (8.0e12 * c.bw * shareP);
                const double tPart =
                    tx * ty * tileBytes * 2.0 * P / kPartialBw + P * tileBytes / kSumBw + 1.0e-6;
                const double tChainP = chain(wgs, std::ceil((double)b.nsteps / P));
                const double cost = bound(std::max(tM, tMemP), tChainP) + tPart;
                if (best.tile < 0 || cost < best.cost) {
                    best.tile = t;
                    best.kind = 2;
                    best.slices = P;
                    best.tMfma = tM;
                    best.tMem = tMemP;
                    best.cost = cost;
                }
            }
            if (best.tile >= 0) ranked.push_back(best);
        }
        // Stream-K tail: when the tiles do not fill the CUs a whole number of
        // times, the CUs that get one tile more set the time, and a wavefront
        // left alone on its SIMD runs slower than two together.  Instead, the
        // tiles of the complete rounds of G = 256 g workgroups run whole and
        // the boxes of the remaining ones are dealt in equal runs to G more
        // workgroups (g = 1 .. the tile's occupancy; the best is kept); the
        // pieces of a tile shared by several of them are summed through the
        // workspace in piece order by the last to finish.  Priced by cu_time
        // for the busiest CU (two boxes of set-up per piece), the partial
        // tiles' traffic (about r + G tile-sized writes and reads, which add
        // about the time of a 6.8 TB/s stream: measured on MI355X, where they
        // overlap the MFMAs of other workgroups) and the last piece's reads of
        // its tile's pieces.
        const double ntile = tx * ty;
        if (c.tail && !(flags & GETT_FLAG_WHOLE_TILES) && !an.emptyC && wpt >= 4 &&
            b.nsteps >= 16 && ntile > 256.0 && std::fmod(ntile, 256.0) > 0.0) {
            const int occ = (int)tail_occupancy(c, itemB);
            const double boxFlops = (double)(c.mt / c.wm) * (c.nt / c.wn) * c.kt * 2.0;
            const double boxTime = std::ceil(wpt / 4.0) * boxFlops / (peakSimd * c.eff) *
                                   (kSplitAhead && c.nbuf == 1 ? 1.4 : 1.0);
            const double tMem = (bytesC + bytesX + bytesY +
                                 0.05 * (bytesX * (ty - 1) + bytesY * (tx - 1))) /
                                (8.0e12 * c.bw);
            Candidate best;
            best.tile = -1;
            for (int g = 1; g <= occ; ++g) {
                const TailShape ts = tail_shape((int64_t)ntile, b.nsteps, 256 * (int64_t)g);
                const double pieces = std::ceil((double)ts.len / b.nsteps) + 1.0;
                const double units = cu_time(occ, (int)std::ceil(ts.full / 256.0), (double)b.nsteps,
                                             (int)std::ceil(ts.wgs / 256.0),
                                             (double)ts.len + 2.0 * pieces);
                const double tM = units * boxTime;
                const double tPart = (double)(ntile - ts.full + ts.wgs) * tileBytes * 2.0 / 6.8e12 +
                                     pieces * tileBytes / kSumBw + 1.0e-6;
                const double cost = bound(std::max(tM, tMem), tChain) + tPart;
                if (best.tile < 0 || cost < best.cost) {
                    best.tile = t;
                    best.kind = 3;
                    best.slices = 256 * g;
                    best.tMfma = tM;
                    best.tMem = tMem;
                    best.cost = cost;
                }
            }
            if (best.tile >= 0) ranked.push_back(best);
        }
    }
    // Ties (the same estimate to 0.01 us: mirror-image tiles on a square
    // problem) between tiles of at least 64 x 64 go to the one wider along y,
    // whose C runs are longer (measured on MI355X: fp64 64 x 128 x 24 against
    // 128 x 64 x 24 on the 4D x 4D contractions of Appendix A, 1-4% faster);
    // small tiles keep the table's order (fp32 64 x 32 was 3-5% faster than
    // 32 x 64 on the latency-bound points of Fig. 11).
    auto wideY = [&](const Candidate &c) {
        const TileShape &t = tile_shape(dtype, c.tile);
        return t.mt >= 64 && t.nt >= 64 ? t.nt : 0;
    };
    std::stable_sort(ranked.begin(), ranked.end(), [&](const Candidate &a, const Candidate &b) {
        const long long ka = llround(a.cost * 1e8), kb = llround(b.cost * 1e8);
        if (ka != kb) return ka < kb;
        return wideY(a) > wideY(b);
    });
    Candidate pick = ranked[0];
    const char *how = "model";
    auto find = [&](int t, int k) -> const Candidate * {
        for (auto &c : ranked)
            if (c.tile == t && c.kind == k) return &c;
        return nullptr;
    };
    // tuning and test hooks; a choice being timed by gett_plan_tune overrides
    // them, a remembered one does not
    if (force && (force->timing || !(ft || fk))) {
        if (const Candidate *c = find(force->tile, force->kind)) {
            pick = *c;
            how = force->source;
        }
    } else if (ft || fk) {
        const int t = ft ? atoi(ft) : pick.tile;
        const int k = fk ? atoi(fk) : 0;
        const Candidate *c = find(t, k);
        if (!c) c = find(t, 0);
        if (c) {
            pick = *c;
            how = "forced";
            // the stream-K tail on any plan of a tile that carries it (the
            // model ranks it only where it may pay)
            if (k == 3 && c->kind == 0 && tile_shape(dtype, t).tail && !an.emptyC &&
                !(flags & GETT_FLAG_WHOLE_TILES))
                pick.kind = 3;
        }
    }
    // tuning hook: this many K slices on the chosen tile
    // (1: none), unless the plan must be deterministic
    if (const char *fs = hk.forceKslices) {
        const int P = atoi(fs);
        if (P == 1 && pick.kind == 2) {
            if (const Candidate *c = find(pick.tile, 0)) pick = *c;
        } else if (P > 1 && pick.kind != 1 && !an.emptyC && !(flags & GETT_FLAG_WHOLE_TILES)) {
            pick.kind = 2;
            pick.slices = P;
        }
    }
    const int tile = pick.tile;
    int kind = pick.kind;
    const int kslices = kind == 2 ? pick.slices : 1;
    const double bestMfma = pick.tMfma, bestMem = pick.tMem;
    const TileShape &ts = tile_shape(dtype, tile);

    // ---- index splitting (Sec. 3.2.1, Fig. 5: the sub-tensors keep the
    //      stride-one index of every tensor; Examples 1-2: one index read as
    //      two).  The tiles are linear ranges of each set in its order, so a
    //      set whose first index is one tensor's stride-one index and whose
    //      second is another's holds both runs only when the first is
    //      blocked: (u, v, ...) becomes (u_in, v, u_out, ...) with u_in of
    //      extent f.  Two cases:
    //        columns -- C's stride-one index u and the column operand's
    //                   stride-one index v are different free indices of
    //                   the column set: C is written in runs of f elements,
    //                   Y is read in 16-byte vectors along v;
    //        K box   -- the row operand's stride-one index u and the column
    //                   operand's v are different contracted indices: X is
    //                   read in vectors along u_in, Y along v.
    //      f is a power of two dividing S_u; the vectors of Y then gather
    //      elements f rows (K positions) apart. ----
    int ysplit = 0;   // 0, kGatherRowVecStrided or kGatherKVecStrided
    int yes = 1;
    if (maySplit) {
        // which set holds each operand's stride-one index
        const int yRow = unit_in(Iy, sY);
        if (yRow > 0 && Iy[0].strC == 1 && Iy[yRow].extent % VW == 0 &&
            (int)Iy.size() < kMaxDims) {
            // Columns.  A tile then writes C in runs of f elements and reads Y
            // in runs of NT/f elements along v; in the whole-index order it
            // writes runs of up to NT along u and reads Y in runs of NT over
            // the extents before v.  Runs are priced per byte: a read run of
            // L bytes at max(1, 64 / L), a write run at max(1, 128 / L)^2
            // (partial lines are far costlier to write than to read: on
            // MI355X, C runs under 64 bytes slowed the column-split
            // contractions of Appendix A 1.4-3.5x, 32-byte read runs did not).
            // f minimises Y's plus C's price; the whole-index order is kept
            // where it is cheaper (a Y that is small next to C).
            const double Ybytes = itemB * (double)sizeY * (double)an.sizeK;
            const double Cbytes = itemB * (double)sizeX * (double)sizeY;
            auto readPrice = [](double L) { return std::max(1.0, 64.0 / L); };
            auto writePrice = [](double L) {
                const double r = std::max(1.0, 128.0 / L);
                return r * r;
            };
            auto runs = [&](double elems, double cap) { return std::max(1.0, std::min(elems, cap)); };
            double before = 1;
            for (int i = 0; i < yRow; ++i) before *= (double)Iy[i].extent;
            const double vExt = (double)Iy[yRow].extent, uExt = (double)Iy[0].extent;
            double best = Ybytes * readPrice(itemB * runs(ts.nt / before, vExt)) +
                          Cbytes * writePrice(itemB * runs(std::min<double>(ts.nt, uExt), uExt));
            int64_t f = 0;
            for (int64_t t = VW; t <= pow2_part(Iy[0].extent) && t * itemB <= 128; t *= 2) {
                if (ts.nt % (t * VW)) continue;
                const double c = Ybytes * readPrice(itemB * runs((double)ts.nt / t, vExt)) +
                                 Cbytes * writePrice(itemB * t);
                if (c < best) { best = c; f = t; }
            }
            if (const char *fs = hk.splitF) f = atoi(fs);   // tuning hook
            std::vector<Index> trial = Iy;
            if (f >= VW && (f & (f - 1)) == 0 && Iy[0].extent % f == 0 && ts.nt % (f * VW) == 0) {
                split_front(trial, 0, (size_t)yRow, f);
                if (aligned(trial, sY, 1) && aligned(Ik, sY, -1)) {
                    Iy.swap(trial);
                    ysplit = kGatherRowVecStrided;
                    yes = (int)f;
                }
            }
        } else {
            std::vector<Index> trial;
            const int64_t f = k_split(ts.kt, trial);
            if (f > 0) {
                Ik.swap(trial);
                nk = (int)Ik.size();
                kvecIdx = 1;
                // the streaming kernel takes the contracted set in one box
                if (kind == 1 && box_for(ts.kt).nsteps > 1) {
                    Ik.swap(trial);
                    nk = (int)Ik.size();
                    kvecIdx = 0;
                } else {
                    ysplit = kGatherKVecStrided;
                    yes = (int)f;
                }
            }
        }
    }
    const Box box = box_for(ts.kt);
    // A contraction bound by the C stream walks C in memory order: x indices
    // by C stride (the row operand's stride-one index stays first when it is
    // a free index, for its vector gathers) and tiles y-fastest.
    const bool streaming = bestMem > bestMfma;
    // C's stride-one run along y, when shorter than a cache line and continued
    // in memory by a row index: C is then stored in its memory order (below),
    // which pays only if consecutive tile rows are consecutive in C, so that
    // row index leads the x order -- taken when the row operand is small next
    // to C (its gathers may lose their vectors).
    const int64_t shortRun = Iy[0].strC == 1 && Iy[0].extent * (int64_t)itemB < 128 ? Iy[0].extent : 0;
    int rowNext = -1;
    for (size_t i = 0; i < Ix.size() && shortRun; ++i)
        if (Ix[i].strC == shortRun) rowNext = (int)i;
    const bool corderRows = rowNext >= 0 && ts.corder && bytesX * 8.0 < bytesC &&
                            !(flags & GETT_FLAG_SCALAR);
    if (streaming) {
        std::stable_sort(Ix.begin(), Ix.end(), [](const Index &a, const Index &b) {
            return a.strC < b.strC;
        });
        for (size_t i = 0; i < Ix.size() && !corderRows; ++i)
            if (sX(Ix[i]) == 1) {
                std::rotate(Ix.begin(), Ix.begin() + i, Ix.begin() + i + 1);
                break;
            }
    } else if (corderRows) {
        std::rotate(Ix.begin(), Ix.begin() + rowNext, Ix.begin() + rowNext + 1);
    }
    const int kj = box.kj;
    const int64_t tj = box.tj, kbox = box.kbox, nblk = box.nblk, nsteps = box.nsteps;

    // ---- gather modes ----
    auto row_vec_ok = [&](const std::vector<Index> &I, auto strOf) {
        if (strOf(I[0]) != 1 || I[0].extent % VW) return false;
        for (size_t i = 1; i < I.size(); ++i)
            if (strOf(I[i]) % VW) return false;
        for (auto &k : Ik)
            if (strOf(k) % VW) return false;
        return true;
    };
    auto k_vec_ok = [&](const std::vector<Index> &I, auto strOf) {
        if (!kvec_ok(strOf)) return false;
        if (kj == 0 && (tj % VW)) return false;
        for (auto &x : I)
            if (strOf(x) % VW) return false;
        return true;
    };
    int xmode = kGatherScalar, ymode = kGatherScalar;
    if (!(flags & GETT_FLAG_SCALAR)) {
        if (row_vec_ok(Ix, sX)) xmode = kGatherRowVec;
        else if (k_vec_ok(Ix, sX)) xmode = kGatherKVec;
        if (ysplit) ymode = ysplit;
        else if (row_vec_ok(Iy, sY)) ymode = kGatherRowVec;
        else if (k_vec_ok(Iy, sY)) ymode = kGatherKVec;
    }
    // The direct-load kernel takes vector gathers of both operands; a plan
    // that ends up otherwise runs its tile's macro-kernel.
    if (kind == 4 && !(xmode <= kGatherKVec && ymode <= kGatherKVec && nsteps >= 1)) kind = 0;
    if (kind == 5 && !(xmode <= kGatherKVec && ymode <= kGatherKVec && nsteps == 1)) kind = 0;
    bool cvec = !(flags & GETT_FLAG_SCALAR) && Iy[0].strC == 1 && Iy[0].extent % VW == 0;
    for (auto &x : Ix) if (x.strC % VW) cvec = false;
    for (size_t i = 1; i < Iy.size(); ++i) if (Iy[i].strC % VW) cvec = false;
    if (ts.ry != VW) cvec = false;   // the tile's lanes do not own VW consecutive columns
    // C stored in its memory order through LDS (unpack_c_order): when C's
    // stride-one run along y is shorter than a cache line and C continues in
    // memory along a row index, the per-lane stores would cut every line.
    // At least one run must fit a staging pass of the packing buffers.
    int crun = 0;
    if (cvec && ts.corder && kind == 0 && kslices == 1 && ysplit != kGatherRowVecStrided &&
        Iy.size() > 1) {
        const int64_t E = Iy[0].extent;
        bool rowNext = false;
        for (auto &x : Ix)
            if (x.strC == E) rowNext = true;
        const int64_t cap = (int64_t)ts.nbuf * ts.kt * ((ts.mt + VW) + (ts.nt + VW));
        if (rowNext && E * (int64_t)itemB < 128 && E % VW == 0 && E < ts.nt &&
            (cap / ts.mt - VW) / E >= 1)
            crun = (int)E;
    }
    if (const char *co = hk.cOrder) {   // tuning hook: 0 turns it off
        if (atoi(co) == 0) crun = 0;
    }

    // ---- addressing: the kernels reach each tile through 64-bit base
    //      offsets and address inside it with 32-bit offsets (rows and
    //      columns relative to the tile's base, K-box positions relative to
    //      the box origin), so tensors may hold 2^31 elements or more as long
    //      as one tile's rows plus one box span less than 2^31 - 1 elements.
    //      Over R consecutive positions of a set, digit i moves at most
    //      min(e_i - 1, floor((R - 1) / P_i) + 1) above its lowest value
    //      (P_i: product of the earlier extents). ----
    {
        constexpr int64_t cap = (int64_t)1 << 62;
        auto sat = [](int64_t a, int64_t b) {   // a * b, saturating at cap
            return (a != 0 && b > cap / a) ? cap : a * b;
        };
        auto span = [&](const std::vector<Index> &I, auto strOf, int64_t R) {
            int64_t tot = 0, P = 1;
            for (const Index &x : I) {
                const int64_t moves = std::min<int64_t>(x.extent - 1, (R - 1) / P + 1);
                tot = std::min(cap, tot + sat(std::max<int64_t>(moves, 0), strOf(x)));
                P = sat(P, std::max<int64_t>(x.extent, 1));
            }
            return tot;
        };
        auto kspan = [&](auto strOf) {
            int64_t tot = sat(box.tj - 1, strOf(Ik[box.kj]));
            for (int i = 0; i < box.kj; ++i)
                tot = std::min(cap, tot + sat(Ik[i].extent - 1, strOf(Ik[i])));
            return tot;
        };
        auto sC = [](const Index &x) { return x.strC; };
        const int64_t lim = INT32_MAX;
        if (!an.emptyC && (span(Ix, sX, ts.mt) + kspan(sX) >= lim ||
                           span(Iy, sY, ts.nt) + kspan(sY) >= lim ||
                           span(Ix, sC, ts.mt) + span(Iy, sC, ts.nt) >= lim))
            return GETT_ERROR_NOT_SUPPORTED;
    }

    // ---- descriptor ----
    KDesc d;
    memset(&d, 0, sizeof(d));
    d.sizeX = sizeX;
    d.sizeY = sizeY;
    d.nx = (int)Ix.size();
    d.ny = (int)Iy.size();
    for (int i = 0; i < d.nx; ++i) {
        d.extX[i] = (int32_t)Ix[i].extent;
        d.strXop[i] = sX(Ix[i]);
        d.strCx[i] = Ix[i].strC;
    }
    for (int i = 0; i < d.ny; ++i) {
        d.extY[i] = (int32_t)Iy[i].extent;
        d.strYop[i] = sY(Iy[i]);
        d.strCy[i] = Iy[i].strC;
    }
    d.nk = nk;
    for (int i = 0; i < nk; ++i) {
        d.extK[i] = (int32_t)Ik[i].extent;
        d.strXk[i] = sX(Ik[i]);
        d.strYk[i] = sY(Ik[i]);
    }
    d.kj = kj;
    d.tj = (int32_t)tj;
    d.kbox = (int32_t)kbox;
    d.nblk = (int32_t)std::max<int64_t>(nblk, 1);
    d.nsteps = nsteps;
    const int64_t tilesX = (sizeX + ts.mt - 1) / ts.mt;
    const int64_t tilesY = (sizeY + ts.nt - 1) / ts.nt;
    if (!an.emptyC && (tilesX * tilesY * ts.wm * ts.wn * 64 >= (int64_t)UINT32_MAX || sizeX >= INT32_MAX ||
                       sizeY >= INT32_MAX || nsteps >= INT32_MAX))
        return GETT_ERROR_NOT_SUPPORTED;
    d.tilesX = (int32_t)tilesX;
    d.tilesY = (int32_t)tilesY;
    d.group = (int32_t)std::max<int64_t>(1, std::min<int64_t>(8, tilesX));
    d.order = streaming ? 1 : 0;
    d.xcdremap = -1;   // decided per call (see gett_contract)
    if (const char *xr = hk.xcdRemap) d.xcdremap = atoi(xr) != 0;   // tuning hook
    d.cvec = cvec ? 1 : 0;
    d.xscalar_kfast = sX(Ik[0]) < sX(Ix[0]) ? 1 : 0;
    d.yscalar_kfast = sY(Ik[0]) < sY(Iy[0]) ? 1 : 0;
    // Element-wise gathers of an operand that is stride-one along the second
    // index of its free set: the lanes walk that index (rows grouped by the
    // first index's value) -- their loads then touch few cache lines.
    auto lane_perm = [&](const std::vector<Index> &I, auto strOf, int mode, int rows,
                         int32_t &kfast) -> int32_t {
        if (mode != kGatherScalar || I.size() < 2 || strOf(I[1]) != 1 || I[0].extent >= rows ||
            I[0].extent < 2)
            return 0;
        kfast = 0;
        return (int32_t)I[0].extent;
    };
    d.xperm = lane_perm(Ix, sX, xmode, ts.mt, d.xscalar_kfast);
    d.yperm = lane_perm(Iy, sY, ymode, ts.nt, d.yscalar_kfast);
    if (const char *lp = hk.lanePerm) {   // tuning hook: 0 turns it off
        if (atoi(lp) == 0) d.xperm = d.yperm = 0;
    }
    d.yes = yes;
    d.kslices = kslices;
    d.crun = crun;
    d.tile0 = 0;
    d.tailFull = d.tailWgs = d.tailLen = 0;
    if (kind == 3 && !an.emptyC) {
        // the model's number of tail workgroups (256 when the tail was forced
        // on a plan the model did not rank it for; tuning hook: GETT_TAIL_WGS)
        int64_t wgs = pick.kind == 3 && pick.slices > 1 ? pick.slices : 256;
        if (const char *tw = hk.tailWgs) wgs = std::max<int64_t>(1, atoll(tw));
        const TailShape tsh = tail_shape((int64_t)tilesX * tilesY, std::max<int64_t>(nsteps, 1), wgs);
        d.tailFull = (int32_t)tsh.full;
        d.tailWgs = (int32_t)tsh.wgs;
        d.tailLen = (int32_t)tsh.len;
    }
    if (!an.emptyC && tilesX * tilesY * kslices * ts.wm * ts.wn * 64 >= (int64_t)UINT32_MAX)
        return GETT_ERROR_NOT_SUPPORTED;
    // Workspace of the partial tiles: a counter per tile that has pieces and
    // a slot per piece (K slices: every slice of every tile; stream-K tail:
    // slots up to (tail workgroups - 1) + (tail tiles - 1), see the kernel).
    int64_t wsSlots = 0, wsCounters = 0;
    if (!an.emptyC) {
        const int64_t tiles = tilesX * tilesY;
        if (kslices > 1) {
            wsSlots = tiles * kslices;
            wsCounters = tiles;
        } else if (kind == 3) {
            wsCounters = tiles - d.tailFull;
            wsSlots = d.tailWgs + wsCounters - 1;
        }
    }
    plan.wsCounters = (uint64_t)wsCounters;
    plan.wsTileBytes = (uint64_t)wsSlots * ts.mt * ts.nt * (dtype == GETT_FLOAT32 ? 4 : 8);

    plan.dtype = dtype;
    plan.flags = flags;
    plan.hooks = hk.text;
    plan.rank[0] = rank[0];
    plan.rank[1] = rank[1];
    plan.rank[2] = rank[2];
    plan.an = an;
    plan.desc = d;
    plan.descScalar = d;
    plan.descScalar.cvec = 0;
    plan.tile = tile;
    plan.xmode = xmode;
    plan.kind = kind;
    plan.ranked = ranked;
    plan.ymode = ymode;
    const double item = dtype == GETT_FLOAT32 ? 4.0 : 8.0;
    plan.flops = 2.0 * (double)an.sizeM * (double)an.sizeN * (double)an.sizeK;
    const double nA = (double)an.sizeM * an.sizeK, nB = (double)an.sizeN * an.sizeK,
                 nC = (double)an.sizeM * an.sizeN;
    plan.bytesAlgo = item * (nA + nB + nC);

    // ---- description ----
    std::ostringstream o;
    o << "{\"dtype\":\"" << (dtype == GETT_FLOAT32 ? "f32" : "f64") << "\",";
    json_set(o, "I_m", an.Im, true, false, true);
    o << ",";
    json_set(o, "I_n", an.In, false, true, true);
    o << ",";
    json_set(o, "I_k", an.Ik, true, true, false);
    o << ",\"merges\":[";
    for (size_t i = 0; i < an.merges.size(); ++i) o << (i ? "," : "") << "\"" << an.merges[i] << "\"";
    o << "],\"swapped\":" << (swap ? "true" : "false");
    o << ",\"row_operand\":\"" << (swap ? "B" : "A") << "\",\"col_operand\":\"" << (swap ? "A" : "B")
      << "\"";
    auto names = [&](const char *key, const std::vector<Index> &s) {
        o << ",\"" << key << "\":[";
        for (size_t i = 0; i < s.size(); ++i) o << (i ? "," : "") << "\"" << s[i].name << "\"";
        o << "]";
    };
    names("x_order", Ix);
    names("y_order", Iy);
    names("k_order", Ik);
    o << ",\"size_x\":" << sizeX << ",\"size_y\":" << sizeY << ",\"size_k\":" << an.sizeK;
    o << ",\"tile\":{\"id\":" << tile << ",\"mt\":" << ts.mt << ",\"nt\":" << ts.nt << ",\"kt\":" << ts.kt
      << ",\"waves\":[" << ts.wm << "," << ts.wn << "],\"reads\":[" << ts.rx << "," << ts.ry
      << "],\"waves_per_simd\":" << ts.wpe << ",\"prefetch\":" << ts.pf
      << ",\"lds_buffers\":" << ts.nbuf << ",\"one_box\":" << (ts.onebox ? "true" : "false")
      << ",\"c_order_epilogue\":" << (ts.corder ? "true" : "false")
      << ",\"chosen_by\":\"" << how << "\",\"model_us\":" << pick.cost * 1e6 << "}";
    o << ",\"hooks\":\"" << hk.text << "\"";
    o << ",\"candidates\":[";
    for (size_t i = 0; i < ranked.size(); ++i) {
        o << (i ? "," : "") << "{\"tile\":" << ranked[i].tile << ",\"kind\":\""
          << kind_name(ranked[i].kind) << "\"";
        if (ranked[i].kind == 2) o << ",\"kslices\":" << ranked[i].slices;
        if (ranked[i].kind == 3) o << ",\"tail_workgroups\":" << ranked[i].slices;
        o << ",\"model_us\":" << ranked[i].cost * 1e6 << "}";
    }
    o << "]";
    o << ",\"streaming\":" << (streaming ? "true" : "false");
    o << ",\"kernel\":\"" << (kind == 2 ? "macro" : kind_name(kind))
      << "\",\"kslices\":" << kslices;
    o << ",\"tail\":{\"full_tiles\":" << d.tailFull << ",\"workgroups\":" << d.tailWgs
      << ",\"boxes\":" << d.tailLen << "}";
    o << ",\"partials\":\"" << (kslices > 1 || kind == 3 ? "workspace" : "none")
      << "\",\"workspace_bytes\":" << plan.wsTileBytes
      << ",\"workspace_counters\":" << plan.wsCounters;
    o << ",\"kbox\":{\"kj\":" << kj << ",\"tj\":" << tj << ",\"elements\":" << kbox << ",\"blocks\":" << nblk
      << ",\"steps\":" << nsteps << "}";
    o << ",\"gather_x\":\"" << mode_name(xmode) << "\",\"gather_y\":\"" << mode_name(ymode)
      << "\",\"c_vector\":" << (cvec ? "true" : "false") << ",\"y_vector_stride\":" << yes
      << ",\"c_order_run\":" << crun << ",\"lane_perm\":[" << d.xperm << "," << d.yperm << "]";
    o << ",\"grid\":{\"tiles_x\":" << tilesX << ",\"tiles_y\":" << tilesY << ",\"workgroups\":"
      << tilesX * tilesY << ",\"threads\":" << ts.wm * ts.wn * 64 << "}";
    o << ",\"empty_c\":" << (an.emptyC ? "true" : "false") << ",\"empty_sum\":"
      << (an.emptySum ? "true" : "false");
    char buf[64];
    snprintf(buf, sizeof buf, "%.17g", plan.flops);
    o << ",\"flops\":" << buf;
    snprintf(buf, sizeof buf, "%.17g", plan.bytesAlgo);
    o << ",\"bytes_min\":" << buf << "}";
    plan.text = o.str();
    return GETT_SUCCESS;
}

}  // namespace gett
