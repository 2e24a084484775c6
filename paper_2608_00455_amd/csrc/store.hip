// Storage-mediated publication of sparse BF16 deltas (paper sec. 4.4,
// cross-cluster transfer): chunk serialisation, Zstandard compression,
// XXH64 checksums, writer parts, the committed manifest and the version
// chain on the host; narrowing of flat offsets to segment-local 32-bit
// indices (writer) and widening back (reader) on the device.
//
// Writer: the ordered delta stays on the device; a bounds kernel finds every
// segment's entry range by binary search, a narrowing kernel turns offsets
// into local indices, and chunks of at most chunk_entries entries move
// through a ring of threads + 2 pinned slots to the host threads, which
// encode, compress, checksum and write them.  Reader: host threads read,
// verify and decode chunks into pinned slots, each slot is copied to the
// device, and a widening kernel restores the flat offsets.
#include <hip/hip_runtime.h>

#include <dirent.h>
#include <dlfcn.h>
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <deque>
#include <functional>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/dte_store.h"
#include "abi_guard.h"

namespace {

// ---- XXH64 (the published 64-bit xxHash algorithm) ------------------------

constexpr uint64_t kP1 = 0x9E3779B185EBCA87ull;
constexpr uint64_t kP2 = 0xC2B2AE3D27D4EB4Full;
constexpr uint64_t kP3 = 0x165667B19E3779F9ull;
constexpr uint64_t kP4 = 0x85EBCA77C2B2AE63ull;
constexpr uint64_t kP5 = 0x27D4EB2F165667C5ull;

inline uint64_t rotl64(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }
inline uint64_t load64(const uint8_t* p)
{
    uint64_t v;
    std::memcpy(&v, p, 8);   // little-endian host (x86-64)
    return v;
}
inline uint32_t load32(const uint8_t* p)
{
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}
inline uint64_t xround(uint64_t acc, uint64_t lane)
{
    acc += lane * kP2;
    acc = rotl64(acc, 31);
    return acc * kP1;
}
inline uint64_t xmerge(uint64_t acc, uint64_t v)
{
    acc ^= xround(0, v);
    return acc * kP1 + kP4;
}

uint64_t xxh64(const void* data, size_t n, uint64_t seed)
{
    const uint8_t* p = static_cast<const uint8_t*>(data);
    const uint8_t* end = p + n;
    uint64_t h;
    if (n >= 32) {
        uint64_t a1 = seed + kP1 + kP2, a2 = seed + kP2, a3 = seed, a4 = seed - kP1;
        const uint8_t* limit = end - 32;
        do {
            a1 = xround(a1, load64(p));
            a2 = xround(a2, load64(p + 8));
            a3 = xround(a3, load64(p + 16));
            a4 = xround(a4, load64(p + 24));
            p += 32;
        } while (p <= limit);
        h = rotl64(a1, 1) + rotl64(a2, 7) + rotl64(a3, 12) + rotl64(a4, 18);
        h = xmerge(h, a1);
        h = xmerge(h, a2);
        h = xmerge(h, a3);
        h = xmerge(h, a4);
    } else {
        h = seed + kP5;
    }
    h += (uint64_t)n;
    while (p + 8 <= end) {
        h ^= xround(0, load64(p));
        h = rotl64(h, 27) * kP1 + kP4;
        p += 8;
    }
    if (p + 4 <= end) {
        h ^= (uint64_t)load32(p) * kP1;
        h = rotl64(h, 23) * kP2 + kP3;
        p += 4;
    }
    while (p < end) {
        h ^= (uint64_t)(*p) * kP5;
        h = rotl64(h, 11) * kP1;
        ++p;
    }
    h ^= h >> 33;
    h *= kP2;
    h ^= h >> 29;
    h *= kP3;
    h ^= h >> 32;
    return h;
}

// ---- Zstandard, loaded at run time from the system library ----------------

struct Zstd {
    size_t (*bound)(size_t) = nullptr;
    size_t (*compress)(void*, size_t, const void*, size_t, int) = nullptr;
    size_t (*decompress)(void*, size_t, const void*, size_t) = nullptr;
    unsigned (*is_error)(size_t) = nullptr;
    bool ok = false;
};

const Zstd& zstd()
{
    static const Zstd z = [] {
        Zstd r;
        void* h = dlopen("libzstd.so.1", RTLD_NOW | RTLD_LOCAL);
        if (!h) return r;
        r.bound = reinterpret_cast<size_t (*)(size_t)>(dlsym(h, "ZSTD_compressBound"));
        r.compress = reinterpret_cast<size_t (*)(void*, size_t, const void*, size_t, int)>(
            dlsym(h, "ZSTD_compress"));
        r.decompress = reinterpret_cast<size_t (*)(void*, size_t, const void*, size_t)>(
            dlsym(h, "ZSTD_decompress"));
        r.is_error = reinterpret_cast<unsigned (*)(size_t)>(dlsym(h, "ZSTD_isError"));
        r.ok = r.bound && r.compress && r.decompress && r.is_error;
        return r;
    }();
    return z;
}

// ---- chunk format -----------------------------------------------------------

constexpr uint32_t kFormat = 1;

struct ChunkHeader {
    char magic[4];          // "DTEC"
    uint32_t format;        // 1
    int32_t segment;
    uint32_t transform;     // 0: indices as values, 1: as gaps
    int64_t first;          // ordinal of the chunk's first entry among its segment's entries
    int64_t count;
    int64_t payload_bytes;  // 6 * count
};
static_assert(sizeof(ChunkHeader) == 40, "chunk header is 40 bytes");

struct ChunkMeta {
    std::string file;
    int32_t writer = 0;
    int32_t segment = 0;
    int64_t first = 0;
    int64_t count = 0;
    int64_t raw_bytes = 0;
    int64_t bytes = 0;
    uint64_t xxh = 0;
};

// Encode `count` ascending local indices and values as a stored chunk.
dte_status encode_chunk(const uint32_t* local, const uint16_t* val, int64_t count, int32_t segment,
                        int64_t first, const dte_store_options& o, std::vector<uint8_t>& out)
{
    const size_t payload = (size_t)count * 6;
    std::vector<uint8_t> raw(payload);
    uint32_t* ri = reinterpret_cast<uint32_t*>(raw.data());
    uint32_t prev = 0;
    for (int64_t i = 0; i < count; ++i) {
        const uint32_t x = local[i];
        ri[i] = o.index_transform == 1 ? x - prev : x;
        prev = x;
    }
    std::memcpy(raw.data() + (size_t)count * 4, val, (size_t)count * 2);
    ChunkHeader h;
    std::memcpy(h.magic, "DTEC", 4);
    h.format = kFormat;
    h.segment = segment;
    h.transform = (uint32_t)o.index_transform;
    h.first = first;
    h.count = count;
    h.payload_bytes = (int64_t)payload;
    if (o.codec == 0) {
        out.resize(sizeof h + payload);
        std::memcpy(out.data(), &h, sizeof h);
        std::memcpy(out.data() + sizeof h, raw.data(), payload);
        return DTE_OK;
    }
    const Zstd& z = zstd();
    if (!z.ok) return DTE_ERR_UNSUPPORTED;
    const size_t cap = z.bound(payload);
    out.resize(sizeof h + cap);
    std::memcpy(out.data(), &h, sizeof h);
    const size_t got = z.compress(out.data() + sizeof h, cap, raw.data(), payload, o.level);
    if (z.is_error(got)) return DTE_ERR_IO;
    out.resize(sizeof h + got);
    return DTE_OK;
}

// Verify and decode a stored chunk against its manifest record; writes the
// local indices and values.
dte_status decode_chunk(const std::vector<uint8_t>& bytes, const ChunkMeta& m, int64_t numel,
                        bool compressed, uint32_t* local, uint16_t* val)
{
    if ((int64_t)bytes.size() != m.bytes || bytes.size() < sizeof(ChunkHeader)) return DTE_ERR_CORRUPT;
    if (xxh64(bytes.data(), bytes.size(), 0) != m.xxh) return DTE_ERR_CORRUPT;
    ChunkHeader h;
    std::memcpy(&h, bytes.data(), sizeof h);
    if (std::memcmp(h.magic, "DTEC", 4) != 0 || h.format != kFormat || h.segment != m.segment ||
        h.first != m.first || h.count != m.count || h.payload_bytes != 6 * m.count ||
        h.transform > 1)
        return DTE_ERR_CORRUPT;
    const size_t payload = (size_t)h.payload_bytes;
    std::vector<uint8_t> raw;
    const uint8_t* src = bytes.data() + sizeof h;
    if (compressed) {
        const Zstd& z = zstd();
        if (!z.ok) return DTE_ERR_UNSUPPORTED;
        raw.resize(payload);
        const size_t got = z.decompress(raw.data(), payload, src, bytes.size() - sizeof h);
        if (z.is_error(got) || got != payload) return DTE_ERR_CORRUPT;
        src = raw.data();
    } else if (bytes.size() - sizeof h != payload) {
        return DTE_ERR_CORRUPT;
    }
    uint64_t x = 0;
    for (int64_t i = 0; i < h.count; ++i) {
        const uint32_t w = load32(src + 4 * i);
        x = h.transform == 1 ? x + w : w;
        // ascending, inside the segment (the first gap may be zero)
        if (x >= (uint64_t)numel || (i > 0 && x <= (uint64_t)local[i - 1])) return DTE_ERR_CORRUPT;
        local[i] = (uint32_t)x;
    }
    std::memcpy(val, src + (size_t)h.count * 4, (size_t)h.count * 2);
    return DTE_OK;
}

// ---- files ------------------------------------------------------------------

std::string vdir(const std::string& dir, int64_t version) { return dir + "/v" + std::to_string(version); }

bool write_atomic(const std::string& path, const void* data, size_t n)
{
    const std::string tmp = path + ".tmp." + std::to_string(getpid()) + "." +
                            std::to_string(std::hash<std::thread::id>()(std::this_thread::get_id()));
    const int fd = ::open(tmp.c_str(), O_WRONLY | O_CREAT | O_TRUNC, 0644);
    if (fd < 0) return false;
    const uint8_t* p = static_cast<const uint8_t*>(data);
    size_t left = n;
    while (left > 0) {
        const ssize_t w = ::write(fd, p, left);
        if (w <= 0) {
            ::close(fd);
            ::unlink(tmp.c_str());
            return false;
        }
        p += w;
        left -= (size_t)w;
    }
    if (::fsync(fd) != 0 || ::close(fd) != 0) {
        ::unlink(tmp.c_str());
        return false;
    }
    return ::rename(tmp.c_str(), path.c_str()) == 0;
}

bool read_file(const std::string& path, std::vector<uint8_t>& out)
{
    FILE* f = std::fopen(path.c_str(), "rb");
    if (!f) return false;
    std::fseek(f, 0, SEEK_END);
    const long n = std::ftell(f);
    std::fseek(f, 0, SEEK_SET);
    if (n < 0) {
        std::fclose(f);
        return false;
    }
    out.resize((size_t)n);
    const size_t got = n ? std::fread(out.data(), 1, (size_t)n, f) : 0;
    std::fclose(f);
    return got == (size_t)n;
}

bool make_dir(const std::string& path) { return ::mkdir(path.c_str(), 0755) == 0 || errno == EEXIST; }

// ---- a small JSON reader / writer for parts and manifests -------------------

struct Json {
    enum Kind { Null, Num, Str, Arr, Obj } kind = Null;
    double num = 0;
    int64_t inum = 0;
    std::string str;
    std::vector<Json> arr;
    std::vector<std::pair<std::string, Json>> obj;
    const Json* get(const char* k) const
    {
        for (const auto& kv : obj)
            if (kv.first == k) return &kv.second;
        return nullptr;
    }
};

struct JsonParser {
    const char* p;
    const char* e;
    bool ok = true;
    void ws()
    {
        while (p < e && (*p == ' ' || *p == '\n' || *p == '\r' || *p == '\t')) ++p;
    }
    bool eat(char c)
    {
        ws();
        if (p < e && *p == c) {
            ++p;
            return true;
        }
        return false;
    }
    std::string string()
    {
        std::string s;
        if (!eat('"')) {
            ok = false;
            return s;
        }
        while (p < e && *p != '"') {
            if (*p == '\\') {   // names are stored without escapes
                ok = false;
                return s;
            }
            s.push_back(*p++);
        }
        if (p >= e) ok = false;
        else ++p;
        return s;
    }
    Json value(int depth)
    {
        Json j;
        ws();
        if (depth > 16 || p >= e) {
            ok = false;
            return j;
        }
        if (*p == '{') {
            ++p;
            j.kind = Json::Obj;
            if (eat('}')) return j;
            do {
                std::string k = string();
                if (!ok || !eat(':')) {
                    ok = false;
                    return j;
                }
                j.obj.emplace_back(k, value(depth + 1));
            } while (ok && eat(','));
            if (!eat('}')) ok = false;
        } else if (*p == '[') {
            ++p;
            j.kind = Json::Arr;
            if (eat(']')) return j;
            do j.arr.push_back(value(depth + 1));
            while (ok && eat(','));
            if (!eat(']')) ok = false;
        } else if (*p == '"') {
            j.kind = Json::Str;
            j.str = string();
        } else if (*p == 'n' && e - p >= 4 && std::strncmp(p, "null", 4) == 0) {
            p += 4;
        } else {
            char* q = nullptr;
            const std::string tok(p, (size_t)std::min<ptrdiff_t>(e - p, 32));
            j.kind = Json::Num;
            j.inum = std::strtoll(tok.c_str(), &q, 10);
            const size_t used = (size_t)(q - tok.c_str());
            if (used == 0) {
                ok = false;
                return j;
            }
            j.num = (double)j.inum;
            p += used;
        }
        return j;
    }
};

bool parse_json(const std::vector<uint8_t>& text, Json& out)
{
    JsonParser ps{reinterpret_cast<const char*>(text.data()),
                  reinterpret_cast<const char*>(text.data()) + text.size()};
    out = ps.value(0);
    ps.ws();
    return ps.ok && ps.p == ps.e && out.kind == Json::Obj;
}

bool int_of(const Json& o, const char* k, int64_t& v)
{
    const Json* j = o.get(k);
    if (!j || j->kind != Json::Num) return false;
    v = j->inum;
    return true;
}

std::string hex64(uint64_t x)
{
    char b[17];
    std::snprintf(b, sizeof b, "%016llx", (unsigned long long)x);
    return b;
}

bool unhex64(const std::string& s, uint64_t& x)
{
    if (s.size() != 16) return false;
    char* q = nullptr;
    x = std::strtoull(s.c_str(), &q, 16);
    return q == s.c_str() + 16;
}

struct Segment {
    std::string name;
    int64_t begin = 0;
    int64_t numel = 0;
};

std::string segments_json(const std::vector<Segment>& segs)
{
    std::string s = "[";
    for (size_t i = 0; i < segs.size(); ++i) {
        s += (i ? ",\n  " : "\n  ");
        s += "{\"name\": \"" + segs[i].name + "\", \"flat_begin\": " + std::to_string(segs[i].begin) +
             ", \"numel\": " + std::to_string(segs[i].numel) + "}";
    }
    return s + "]";
}

std::string chunk_json(const ChunkMeta& c)
{
    return "{\"file\": \"" + c.file + "\", \"writer\": " + std::to_string(c.writer) +
           ", \"segment\": " + std::to_string(c.segment) + ", \"first\": " + std::to_string(c.first) +
           ", \"count\": " + std::to_string(c.count) + ", \"raw_bytes\": " +
           std::to_string(c.raw_bytes) + ", \"bytes\": " + std::to_string(c.bytes) +
           ", \"xxh64\": \"" + hex64(c.xxh) + "\"}";
}

bool parse_segments(const Json* a, std::vector<Segment>& out)
{
    if (!a || a->kind != Json::Arr) return false;
    out.clear();
    for (const Json& j : a->arr) {
        Segment s;
        const Json* n = j.get("name");
        if (!n || n->kind != Json::Str || !int_of(j, "flat_begin", s.begin) ||
            !int_of(j, "numel", s.numel))
            return false;
        s.name = n->str;
        out.push_back(s);
    }
    return true;
}

bool parse_chunks(const Json* a, std::vector<ChunkMeta>& out)
{
    if (!a || a->kind != Json::Arr) return false;
    out.clear();
    for (const Json& j : a->arr) {
        ChunkMeta c;
        int64_t w = 0, s = 0;
        const Json* f = j.get("file");
        const Json* x = j.get("xxh64");
        if (!f || f->kind != Json::Str || !x || x->kind != Json::Str || !int_of(j, "writer", w) ||
            !int_of(j, "segment", s) || !int_of(j, "first", c.first) || !int_of(j, "count", c.count) ||
            !int_of(j, "raw_bytes", c.raw_bytes) || !int_of(j, "bytes", c.bytes) ||
            !unhex64(x->str, c.xxh))
            return false;
        if (f->str.find('/') != std::string::npos || f->str.empty()) return false;
        c.file = f->str;
        c.writer = (int32_t)w;
        c.segment = (int32_t)s;
        out.push_back(c);
    }
    return true;
}

bool valid_segments(const std::vector<Segment>& segs)
{
    int64_t end = 0;
    for (const Segment& s : segs) {
        if (s.begin < end || s.numel <= 0 || s.numel > ((int64_t)1 << 32) ||
            s.begin > INT64_MAX - s.numel)
            return false;
        for (char c : s.name)
            if (c == '"' || c == '\\' || (unsigned char)c < 0x20) return false;
        end = s.begin + s.numel;
    }
    return true;
}

bool options_ok(const dte_store_options* o)
{
    return o && (o->codec == 0 || o->codec == 1) && (o->codec == 0 || (o->level >= 1 && o->level <= 19)) &&
           o->threads >= 1 && o->threads <= 64 && (o->index_transform == 0 || o->index_transform == 1) &&
           o->chunk_entries >= 1 && o->chunk_entries <= ((int64_t)1 << 26);
}

// First status other than DTE_OK reported by any thread.
struct FirstError {
    std::mutex m;
    dte_status st = DTE_OK;
    void set(dte_status s)
    {
        std::lock_guard<std::mutex> g(m);
        if (st == DTE_OK) st = s;
    }
    dte_status get()
    {
        std::lock_guard<std::mutex> g(m);
        return st;
    }
};

// ---- a fixed pool of host threads -------------------------------------------

// A job that throws reports DTE_ERR_HOST to `err`; if a thread cannot be
// started, the threads already running are joined before the constructor
// rethrows.
class Pool {
public:
    Pool(int n, FirstError& err) : err_(err)
    {
        try {
            for (int i = 0; i < n; ++i) th_.emplace_back([this] { loop(); });
        } catch (...) {
            finish();
            throw;
        }
    }
    ~Pool() { finish(); }
    void push(std::function<void()> f)
    {
        {
            std::lock_guard<std::mutex> g(m_);
            q_.push_back(std::move(f));
        }
        cv_.notify_one();
    }

private:
    void loop()
    {
        for (;;) {
            std::function<void()> f;
            {
                std::unique_lock<std::mutex> g(m_);
                cv_.wait(g, [this] { return stop_ || !q_.empty(); });
                if (q_.empty()) return;
                f = std::move(q_.front());
                q_.pop_front();
            }
            try {
                f();
            } catch (...) {
                err_.set(DTE_ERR_HOST);
            }
        }
    }
    void finish()
    {
        {
            std::lock_guard<std::mutex> g(m_);
            stop_ = true;
        }
        cv_.notify_all();
        for (auto& t : th_) t.join();
        th_.clear();
    }
    FirstError& err_;
    std::vector<std::thread> th_;
    std::deque<std::function<void()>> q_;
    std::mutex m_;
    std::condition_variable cv_;
    bool stop_ = false;
};

// Slots of pinned host memory handed between the copying thread and the pool.
class Ring {
public:
    Ring(int slots, int64_t entries) : entries_(entries)
    {
        for (int i = 0; i < slots; ++i) {
            void* p = nullptr;
            if (hipHostMalloc(&p, (size_t)entries * 6, hipHostMallocDefault) != hipSuccess) {
                ok_ = false;
                break;
            }
            mem_.push_back(p);
            free_.push_back(i);
        }
    }
    ~Ring()
    {
        for (void* p : mem_) (void)hipHostFree(p);
    }
    bool ok() const { return ok_; }
    int acquire()
    {
        std::unique_lock<std::mutex> g(m_);
        cv_.wait(g, [this] { return !free_.empty(); });
        const int s = free_.back();
        free_.pop_back();
        return s;
    }
    void release(int s)
    {
        {
            std::lock_guard<std::mutex> g(m_);
            free_.push_back(s);
        }
        cv_.notify_one();
    }
    uint32_t* local(int s) { return static_cast<uint32_t*>(mem_[s]); }
    uint16_t* val(int s) { return reinterpret_cast<uint16_t*>(static_cast<uint32_t*>(mem_[s]) + entries_); }

private:
    int64_t entries_;
    std::vector<void*> mem_;
    std::vector<int> free_;
    std::mutex m_;
    std::condition_variable cv_;
    bool ok_ = true;
};

// ---- device kernels ---------------------------------------------------------

__device__ __forceinline__ int64_t lower_bound_i64(const int64_t* a, int64_t n, int64_t x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (a[mid] < x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// lo[s] / hi[s]: first entry at or after the start / end of segment s.
__global__ void bounds_kernel(const int64_t* idx, int64_t n, const int64_t* begin,
                              const int64_t* end, int32_t nseg, int64_t* lo, int64_t* hi)
{
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s < nseg) {
        lo[s] = lower_bound_i64(idx, n, begin[s]);
        hi[s] = lower_bound_i64(idx, n, end[s]);
    }
}

// *bad = 1 if some entry is not above its predecessor.
__global__ void ascending_kernel(const int64_t* idx, int64_t n, int32_t* bad)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    bool ok = true;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x + 1; e < n; e += stride)
        ok = ok && idx[e] > idx[e - 1];
    if (!ok) atomicOr(bad, 1);
}

// A contiguous range [begin, end) of the writer's flat shard holding whole
// rows of a box of canonical segment `segment` (see dte_store_piece).
struct Piece {
    int64_t begin, end;
    int32_t segment;          // -1: not published by this writer
    int64_t local_cols, canon_cols, row0, col0;
};

__host__ __device__ inline int64_t canon_local(const Piece& pc, int64_t q)
{
    if (pc.local_cols == pc.canon_cols && pc.col0 == 0) return pc.row0 * pc.canon_cols + q;
    const int64_t row = q / pc.local_cols;
    return (pc.row0 + row) * pc.canon_cols + pc.col0 + (q - row * pc.local_cols);
}

// local[e]: canonical segment-local index of entry e, from the piece holding
// it (entries already checked to lie inside pieces; pieces sorted by begin).
__global__ void narrow_kernel(const int64_t* idx, int64_t n, const int64_t* begin,
                              const Piece* pieces, int32_t npiece, uint32_t* local)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const int64_t x = idx[e];
        const int64_t k = lower_bound_i64(begin, npiece, x + 1) - 1;   // last begin <= x
        local[e] = k >= 0 ? (uint32_t)canon_local(pieces[k], x - pieces[k].begin) : 0u;
    }
}

// idx[e] = base[c] + local[e] for the chunk c holding entry e (chunk c
// starts at entry first[c]; first[0] == 0, ascending).
__global__ void widen_kernel(const uint32_t* local, int64_t n, const int64_t* first,
                             const int64_t* base, int32_t nchunk, int64_t* idx)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const int64_t c = lower_bound_i64(first, nchunk, e + 1) - 1;
        idx[e] = (c >= 0 ? base[c] : 0) + (int64_t)local[e];
    }
}

// Device allocation released at scope exit.
struct DevBuf {
    void* p = nullptr;
    ~DevBuf()
    {
        if (p) (void)hipFree(p);
    }
    bool alloc(size_t n) { return hipMalloc(&p, n ? n : 8) == hipSuccess; }
};

int device_cus()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 256;
    return cus;
}

std::vector<Segment> to_segments(const dte_store_segment* segs, int32_t nseg)
{
    std::vector<Segment> out((size_t)nseg);
    for (int32_t i = 0; i < nseg; ++i) {
        out[i].name = segs[i].name ? segs[i].name : "";
        out[i].begin = segs[i].flat_begin;
        out[i].numel = segs[i].numel;
    }
    return out;
}

// One chunk to encode: entries [lo, lo + count) of the writer's delta, all
// in piece `piece` of canonical segment `segment`, `first` entries of this
// writer in the segment before it.
struct ChunkJob {
    int32_t segment;
    int32_t piece;
    int64_t lo;
    int64_t first;
    int64_t count;
};

std::vector<ChunkJob> plan_chunks(const std::vector<Piece>& pcs, const std::vector<int64_t>& lo,
                                  const std::vector<int64_t>& hi, int64_t chunk_entries)
{
    std::vector<ChunkJob> jobs;
    std::map<int32_t, int64_t> ordinal;
    for (size_t k = 0; k < pcs.size(); ++k) {
        if (pcs[k].segment < 0) continue;
        int64_t& first = ordinal[pcs[k].segment];
        for (int64_t a = lo[k]; a < hi[k]; a += chunk_entries) {
            const int64_t c = std::min(chunk_entries, hi[k] - a);
            jobs.push_back({pcs[k].segment, (int32_t)k, a, first, c});
            first += c;
        }
    }
    return jobs;
}

// Pieces sorted and disjoint in the shard; each owned piece a whole-row box
// inside its segment; the owned pieces of one segment in ascending, disjoint
// canonical order (so each writer's entries of a segment ascend).
bool valid_pieces(const std::vector<Piece>& pcs, const std::vector<Segment>& segs)
{
    int64_t end = INT64_MIN;
    std::map<int32_t, int64_t> last;   // per segment: largest canonical index so far
    for (const Piece& pc : pcs) {
        if (pc.begin < end || pc.end < pc.begin || pc.begin < 0) return false;
        end = pc.end;
        if (pc.segment < 0) continue;
        if ((size_t)pc.segment >= segs.size() || pc.local_cols <= 0 || pc.canon_cols <= 0 ||
            pc.row0 < 0 || pc.col0 < 0 || pc.col0 + pc.local_cols > pc.canon_cols ||
            (pc.end - pc.begin) % pc.local_cols != 0)
            return false;
        const int64_t rows = (pc.end - pc.begin) / pc.local_cols;
        if (rows == 0) continue;
        const int64_t numel = segs[pc.segment].numel;
        if (pc.canon_cols > numel || pc.row0 + rows > numel / pc.canon_cols ||
            numel % pc.canon_cols != 0)
            return false;
        const int64_t lo = canon_local(pc, 0), hi = canon_local(pc, pc.end - pc.begin - 1);
        auto it = last.find(pc.segment);
        if (it != last.end() && lo <= it->second) return false;
        last[pc.segment] = hi;
    }
    return true;
}

std::vector<Piece> identity_pieces(const std::vector<Segment>& segs)
{
    std::vector<Piece> pcs;
    for (size_t i = 0; i < segs.size(); ++i)
        pcs.push_back({segs[i].begin, segs[i].begin + segs[i].numel, (int32_t)i, segs[i].numel,
                       segs[i].numel, 0, 0});
    return pcs;
}

std::vector<Piece> to_pieces(const dte_store_piece* p, int32_t n)
{
    std::vector<Piece> pcs((size_t)n);
    for (int32_t i = 0; i < n; ++i)
        pcs[i] = {p[i].sender_begin, p[i].sender_end, p[i].segment, p[i].local_cols, p[i].canon_cols,
                  p[i].canon_row0, p[i].canon_col0};
    return pcs;
}

dte_status write_part_file(const std::string& dir, int64_t version, int32_t writer,
                           const std::vector<Segment>& segs, const dte_store_options& o,
                           std::vector<ChunkMeta>& chunks, int64_t entries)
{
    std::sort(chunks.begin(), chunks.end(), [](const ChunkMeta& a, const ChunkMeta& b) {
        return a.segment != b.segment ? a.segment < b.segment : a.first < b.first;
    });
    std::string s = "{\"version\": " + std::to_string(version) + ", \"writer\": " +
                    std::to_string(writer) + ", \"codec\": \"" + (o.codec ? "zstd" : "none") +
                    "\", \"entries\": " + std::to_string(entries) + ",\n\"segments\": " +
                    segments_json(segs) + ",\n\"chunks\": [";
    for (size_t i = 0; i < chunks.size(); ++i) s += (i ? ",\n  " : "\n  ") + chunk_json(chunks[i]);
    s += "]}\n";
    const std::string path = vdir(dir, version) + "/part-" + std::to_string(writer) + ".json";
    return write_atomic(path, s.data(), s.size()) ? DTE_OK : DTE_ERR_IO;
}

// Encode, compress, checksum and write one chunk (host thread).
void encode_and_write(const std::string& vd, int32_t writer, int64_t k, const ChunkJob& j,
                      const uint32_t* local, const uint16_t* val, const dte_store_options& o,
                      std::mutex& mm, std::vector<ChunkMeta>& metas, FirstError& err)
{
    std::vector<uint8_t> bytes;
    const dte_status st = encode_chunk(local, val, j.count, j.segment, j.first, o, bytes);
    if (st != DTE_OK) {
        err.set(st);
        return;
    }
    ChunkMeta c;
    c.file = "chunk-" + std::to_string(writer) + "-" + std::to_string(k) + ".dte";
    c.writer = writer;
    c.segment = j.segment;
    c.first = j.first;
    c.count = j.count;
    c.raw_bytes = 6 * j.count;
    c.bytes = (int64_t)bytes.size();
    c.xxh = xxh64(bytes.data(), bytes.size(), 0);
    if (!write_atomic(vd + "/" + c.file, bytes.data(), bytes.size())) {
        err.set(DTE_ERR_IO);
        return;
    }
    std::lock_guard<std::mutex> g(mm);
    metas.push_back(c);
}

void fill_stats(dte_store_stats* stats, const std::vector<ChunkMeta>& metas)
{
    if (!stats) return;
    std::memset(stats, 0, sizeof *stats);
    for (const ChunkMeta& c : metas) {
        stats->entries += c.count;
        stats->chunks += 1;
        stats->raw_bytes += c.raw_bytes;
        stats->stored_bytes += c.bytes;
    }
}

bool common_write_args(const char* dir, int64_t version, int32_t writer,
                       const dte_store_segment* segs, int32_t nseg, const dte_store_options* opt)
{
    if (!dir || version < 1 || writer < 0 || writer > 4095 || nseg < 0 || (nseg > 0 && !segs) ||
        !options_ok(opt))
        return false;
    return valid_segments(to_segments(segs, nseg));
}

// ---- manifest reading -------------------------------------------------------

struct Manifest {
    int64_t version = 0, parent = 0, entries = 0;
    bool compressed = false;
    std::vector<Segment> segs;
    std::vector<ChunkMeta> chunks;   // ordered by (segment, first)
    std::vector<int64_t> offset;     // entry position of each chunk
};

dte_status load_manifest(const std::string& dir, int64_t version, Manifest& m)
{
    std::vector<uint8_t> text;
    if (!read_file(vdir(dir, version) + "/manifest.json", text)) return DTE_ERR_IO;
    Json j;
    if (!parse_json(text, j)) return DTE_ERR_CORRUPT;
    const Json* codec = j.get("codec");
    if (!int_of(j, "version", m.version) || !int_of(j, "parent", m.parent) ||
        !int_of(j, "entries", m.entries) || !codec || codec->kind != Json::Str ||
        !parse_segments(j.get("segments"), m.segs) || !parse_chunks(j.get("chunks"), m.chunks) ||
        m.version != version || !valid_segments(m.segs))
        return DTE_ERR_CORRUPT;
    if (codec->str != "zstd" && codec->str != "none") return DTE_ERR_CORRUPT;
    m.compressed = codec->str == "zstd";
    int64_t pos = 0;
    for (size_t i = 0; i < m.chunks.size(); ++i) {
        const ChunkMeta& c = m.chunks[i];
        if (c.segment < 0 || (size_t)c.segment >= m.segs.size() || c.count <= 0 ||
            c.count > ((int64_t)1 << 26) || c.raw_bytes != 6 * c.count || c.bytes < 40)
            return DTE_ERR_CORRUPT;
        // ascending (segment, writer); within one, consecutive entry ranges from 0
        const bool same = i > 0 && m.chunks[i - 1].segment == c.segment &&
                          m.chunks[i - 1].writer == c.writer;
        if (i > 0) {
            const ChunkMeta& p = m.chunks[i - 1];
            if (c.segment < p.segment || (c.segment == p.segment && c.writer < p.writer))
                return DTE_ERR_CORRUPT;
        }
        if (c.first != (same ? m.chunks[i - 1].first + m.chunks[i - 1].count : 0))
            return DTE_ERR_CORRUPT;
        m.offset.push_back(pos);
        pos += c.count;
    }
    if (pos != m.entries) return DTE_ERR_CORRUPT;
    return DTE_OK;
}

// Shared reader: verify and decode every chunk on `threads` host threads;
// `sink(chunk, local, val)` receives each decoded chunk (called from the
// pool threads, one chunk at a time per call).
dte_status read_chunks(const std::string& dir, const Manifest& m, int32_t threads,
                       const std::function<dte_status(size_t, const uint32_t*, const uint16_t*)>& sink)
{
    FirstError err;
    {
        Pool pool(threads, err);
        for (size_t k = 0; k < m.chunks.size(); ++k) {
            pool.push([&, k] {
                if (err.get() != DTE_OK) return;
                const ChunkMeta& c = m.chunks[k];
                std::vector<uint8_t> bytes;
                if (!read_file(vdir(dir, m.version) + "/" + c.file, bytes)) {
                    err.set(DTE_ERR_IO);
                    return;
                }
                std::vector<uint32_t> local((size_t)c.count);
                std::vector<uint16_t> v((size_t)c.count);
                const dte_status st =
                    decode_chunk(bytes, c, m.segs[c.segment].numel, m.compressed, local.data(), v.data());
                if (st != DTE_OK) {
                    err.set(st);
                    return;
                }
                const dte_status ss = sink(k, local.data(), v.data());
                if (ss != DTE_OK) err.set(ss);
            });
        }
    }
    return err.get();
}

void read_stats(dte_store_stats* stats, const Manifest& m)
{
    if (!stats) return;
    std::memset(stats, 0, sizeof *stats);
    for (const ChunkMeta& c : m.chunks) {
        stats->entries += c.count;
        stats->chunks += 1;
        stats->raw_bytes += c.raw_bytes;
        stats->stored_bytes += c.bytes;
    }
}

}  // namespace

// ---- C ABI ------------------------------------------------------------------

extern "C" {

uint64_t dte_store_xxh64(const void* data, int64_t n, uint64_t seed)
{
    if (n < 0 || (n > 0 && !data)) return 0;
    return xxh64(data, (size_t)n, seed);
}

}  // extern "C"

namespace {

dte_status write_host_impl(const char* dir, int64_t version, int32_t writer,
                           const std::vector<Segment>& sg, const std::vector<Piece>& pcs,
                           const int64_t* idx, const uint16_t* val, int64_t count,
                           const dte_store_options* opt, dte_store_stats* stats)
{
    if (count < 0 || (count > 0 && (!idx || !val)) || !valid_pieces(pcs, sg)) return DTE_ERR_ARG;
    if (opt->codec == 1 && !zstd().ok) return DTE_ERR_UNSUPPORTED;
    // entries strictly ascending and inside pieces
    for (int64_t e = 1; e < count; ++e)
        if (idx[e] <= idx[e - 1]) return DTE_ERR_ARG;
    std::vector<int64_t> lo(pcs.size()), hi(pcs.size());
    int64_t inside = 0;
    for (size_t k = 0; k < pcs.size(); ++k) {
        lo[k] = std::lower_bound(idx, idx + count, pcs[k].begin) - idx;
        hi[k] = std::lower_bound(idx, idx + count, pcs[k].end) - idx;
        inside += hi[k] - lo[k];
    }
    if (inside != count) return DTE_ERR_ARG;
    const std::string d(dir);
    if (!make_dir(d) || !make_dir(vdir(d, version))) return DTE_ERR_IO;
    const std::vector<ChunkJob> jobs = plan_chunks(pcs, lo, hi, opt->chunk_entries);
    std::vector<ChunkMeta> metas;
    std::mutex mm;
    FirstError err;
    int64_t published = 0;
    for (const ChunkJob& j : jobs) published += j.count;
    {
        Pool pool(opt->threads, err);
        for (size_t k = 0; k < jobs.size(); ++k) {
            pool.push([&, k] {
                const ChunkJob& j = jobs[k];
                const Piece& pc = pcs[j.piece];
                std::vector<uint32_t> local((size_t)j.count);
                for (int64_t i = 0; i < j.count; ++i)
                    local[i] = (uint32_t)canon_local(pc, idx[j.lo + i] - pc.begin);
                encode_and_write(vdir(d, version), writer, (int64_t)k, j, local.data(), val + j.lo, *opt,
                                 mm, metas, err);
            });
        }
    }
    if (err.get() != DTE_OK) return err.get();
    fill_stats(stats, metas);
    return write_part_file(d, version, writer, sg, *opt, metas, published);
}

dte_status write_device_impl(const char* dir, int64_t version, int32_t writer,
                             const std::vector<Segment>& sg, const std::vector<Piece>& pcs,
                             const int64_t* idx, const uint16_t* val, const int64_t* count,
                             int64_t capacity, const dte_store_options* opt, dte_store_stats* stats,
                             void* stream)
{
    if (!count || capacity < 0 || !valid_pieces(pcs, sg)) return DTE_ERR_ARG;
    if (opt->codec == 1 && !zstd().ok) return DTE_ERR_UNSUPPORTED;
    const hipStream_t s = (hipStream_t)stream;
    int64_t n = 0;
    if (hipMemcpyAsync(&n, count, sizeof n, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return DTE_ERR_HIP;
    if (n < 0 || n > capacity || (n > 0 && (!idx || !val))) return DTE_ERR_ARG;
    const std::string d(dir);
    if (!make_dir(d) || !make_dir(vdir(d, version))) return DTE_ERR_IO;
    std::vector<ChunkMeta> metas;
    const int32_t npc = (int32_t)pcs.size();
    if (n == 0 || npc == 0) {
        if (n > 0) return DTE_ERR_ARG;   // entries but no piece to hold them
        fill_stats(stats, metas);
        return write_part_file(d, version, writer, sg, *opt, metas, 0);
    }
    // piece bounds of the ordered delta, and canonical local indices, on the device
    std::vector<int64_t> hb((size_t)npc), he((size_t)npc);
    for (int32_t i = 0; i < npc; ++i) {
        hb[i] = pcs[i].begin;
        he[i] = pcs[i].end;
    }
    DevBuf dbeg, dend, dlo, dhi, dlocal, dbad, dpcs;
    const size_t sb = (size_t)npc * sizeof(int64_t);
    if (!dbeg.alloc(sb) || !dend.alloc(sb) || !dlo.alloc(sb) || !dhi.alloc(sb) ||
        !dlocal.alloc((size_t)n * sizeof(uint32_t)) || !dbad.alloc(sizeof(int32_t)) ||
        !dpcs.alloc((size_t)npc * sizeof(Piece)))
        return DTE_ERR_HIP;
    int32_t* bad = static_cast<int32_t*>(dbad.p);
    const int32_t zero = 0;
    int64_t* b = static_cast<int64_t*>(dbeg.p);
    int64_t* en = static_cast<int64_t*>(dend.p);
    int64_t* lo_d = static_cast<int64_t*>(dlo.p);
    int64_t* hi_d = static_cast<int64_t*>(dhi.p);
    uint32_t* loc = static_cast<uint32_t*>(dlocal.p);
    Piece* pd = static_cast<Piece*>(dpcs.p);
    if (hipMemcpyAsync(bad, &zero, sizeof zero, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(b, hb.data(), sb, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(en, he.data(), sb, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(pd, pcs.data(), (size_t)npc * sizeof(Piece), hipMemcpyHostToDevice, s) !=
            hipSuccess)
        return DTE_ERR_HIP;
    hipLaunchKernelGGL(bounds_kernel, dim3((unsigned)((npc + 255) / 256)), dim3(256), 0, s, idx, n, b,
                       en, npc, lo_d, hi_d);
    const int64_t want = (n + 255) / 256;
    const int64_t cap = (int64_t)device_cus() * 8;
    hipLaunchKernelGGL(narrow_kernel, dim3((unsigned)std::min(want, cap)), dim3(256), 0, s, idx, n, b,
                       pd, npc, loc);
    hipLaunchKernelGGL(ascending_kernel, dim3((unsigned)std::min(want, cap)), dim3(256), 0, s, idx, n,
                       bad);
    std::vector<int64_t> lo((size_t)npc), hi((size_t)npc);
    int32_t unordered = 0;
    if (hipGetLastError() != hipSuccess ||
        hipMemcpyAsync(lo.data(), lo_d, sb, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(hi.data(), hi_d, sb, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(&unordered, bad, sizeof unordered, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return DTE_ERR_HIP;
    if (unordered) return DTE_ERR_ARG;     // not the output of an ordered extract
    int64_t inside = 0;
    for (int32_t i = 0; i < npc; ++i) inside += hi[i] - lo[i];
    if (inside != n) return DTE_ERR_ARG;   // entries outside every piece
    const std::vector<ChunkJob> jobs = plan_chunks(pcs, lo, hi, opt->chunk_entries);
    int64_t biggest = 1, published = 0;
    for (const ChunkJob& j : jobs) {
        biggest = std::max(biggest, j.count);
        published += j.count;
    }
    Ring ring(opt->threads + 2, biggest);
    if (!ring.ok()) return DTE_ERR_HIP;
    std::mutex mm;
    FirstError err;
    {
        Pool pool(opt->threads, err);
        for (size_t k = 0; k < jobs.size() && err.get() == DTE_OK; ++k) {
            const ChunkJob j = jobs[k];
            const int slot = ring.acquire();
            if (hipMemcpyAsync(ring.local(slot), loc + j.lo, (size_t)j.count * 4, hipMemcpyDeviceToHost,
                               s) != hipSuccess ||
                hipMemcpyAsync(ring.val(slot), val + j.lo, (size_t)j.count * 2, hipMemcpyDeviceToHost,
                               s) != hipSuccess ||
                hipStreamSynchronize(s) != hipSuccess) {
                err.set(DTE_ERR_HIP);
                ring.release(slot);
                break;
            }
            pool.push([&, j, k, slot] {
                encode_and_write(vdir(d, version), writer, (int64_t)k, j, ring.local(slot), ring.val(slot),
                                 *opt, mm, metas, err);
                ring.release(slot);
            });
        }
    }
    if (err.get() != DTE_OK) return err.get();
    fill_stats(stats, metas);
    return write_part_file(d, version, writer, sg, *opt, metas, published);
}

}  // namespace

extern "C" {

dte_status dte_store_write_part_host(const char* dir, int64_t version, int32_t writer,
                                     const dte_store_segment* segs, int32_t nseg,
                                     const int64_t* idx, const uint16_t* val, int64_t count,
                                     const dte_store_options* opt, dte_store_stats* stats)
{
    return dte::no_throw([&]() -> dte_status {
        if (!common_write_args(dir, version, writer, segs, nseg, opt)) return DTE_ERR_ARG;
        const std::vector<Segment> sg = to_segments(segs, nseg);
        return write_host_impl(dir, version, writer, sg, identity_pieces(sg), idx, val, count, opt, stats);
    });
}

dte_status dte_store_write_part_host_mapped(const char* dir, int64_t version, int32_t writer,
                                            const dte_store_segment* segs, int32_t nseg,
                                            const dte_store_piece* pieces, int32_t npiece,
                                            const int64_t* idx, const uint16_t* val, int64_t count,
                                            const dte_store_options* opt, dte_store_stats* stats)
{
    return dte::no_throw([&]() -> dte_status {
        if (!common_write_args(dir, version, writer, segs, nseg, opt) || npiece < 0 ||
            (npiece > 0 && !pieces))
            return DTE_ERR_ARG;
        return write_host_impl(dir, version, writer, to_segments(segs, nseg), to_pieces(pieces, npiece),
                               idx, val, count, opt, stats);
    });
}

dte_status dte_store_write_part_device(const char* dir, int64_t version, int32_t writer,
                                       const dte_store_segment* segs, int32_t nseg,
                                       const int64_t* idx, const uint16_t* val,
                                       const int64_t* count, int64_t capacity,
                                       const dte_store_options* opt, dte_store_stats* stats,
                                       void* stream)
{
    return dte::no_throw([&]() -> dte_status {
        if (!common_write_args(dir, version, writer, segs, nseg, opt)) return DTE_ERR_ARG;
        const std::vector<Segment> sg = to_segments(segs, nseg);
        return write_device_impl(dir, version, writer, sg, identity_pieces(sg), idx, val, count, capacity,
                                 opt, stats, stream);
    });
}

dte_status dte_store_write_part_device_mapped(const char* dir, int64_t version, int32_t writer,
                                              const dte_store_segment* segs, int32_t nseg,
                                              const dte_store_piece* pieces, int32_t npiece,
                                              const int64_t* idx, const uint16_t* val,
                                              const int64_t* count, int64_t capacity,
                                              const dte_store_options* opt, dte_store_stats* stats,
                                              void* stream)
{
    return dte::no_throw([&]() -> dte_status {
        if (!common_write_args(dir, version, writer, segs, nseg, opt) || npiece < 0 ||
            (npiece > 0 && !pieces))
            return DTE_ERR_ARG;
        return write_device_impl(dir, version, writer, to_segments(segs, nseg), to_pieces(pieces, npiece),
                                 idx, val, count, capacity, opt, stats, stream);
    });
}

dte_status dte_store_commit(const char* dir, int64_t version, int64_t parent, int32_t nwriters,
                            int32_t* committed)
{
    return dte::no_throw([&]() -> dte_status {
        if (!dir || version < 1 || parent < 0 || parent >= version || nwriters < 1 || nwriters > 4096 ||
            !committed)
            return DTE_ERR_ARG;
        *committed = 0;
        const std::string d(dir), vd = vdir(d, version);
        std::vector<Segment> segs;
        std::vector<ChunkMeta> chunks;
        std::string codec;
        int64_t entries = 0;
        for (int32_t w = 0; w < nwriters; ++w) {
            std::vector<uint8_t> text;
            if (!read_file(vd + "/part-" + std::to_string(w) + ".json", text)) return DTE_ERR_IO;
            Json j;
            int64_t v = 0, wr = 0, e = 0;
            std::vector<Segment> ps;
            std::vector<ChunkMeta> pc;
            const Json* c = nullptr;
            if (!parse_json(text, j) || !int_of(j, "version", v) || !int_of(j, "writer", wr) ||
                !int_of(j, "entries", e) || !(c = j.get("codec")) || c->kind != Json::Str ||
                !parse_segments(j.get("segments"), ps) || !parse_chunks(j.get("chunks"), pc) ||
                v != version || wr != w)
                return DTE_ERR_CORRUPT;
            if (w == 0) {
                segs = ps;
                codec = c->str;
            } else {
                if (c->str != codec || ps.size() != segs.size()) return DTE_ERR_ARG;
                for (size_t i = 0; i < ps.size(); ++i)
                    if (ps[i].name != segs[i].name || ps[i].begin != segs[i].begin ||
                        ps[i].numel != segs[i].numel)
                        return DTE_ERR_ARG;
            }
            int64_t sum = 0;
            for (const ChunkMeta& m : pc) sum += m.count;
            if (sum != e) return DTE_ERR_CORRUPT;
            entries += e;
            chunks.insert(chunks.end(), pc.begin(), pc.end());
        }
        if (entries == 0) {   // no changed payload anywhere: no new version
            if (DIR* dd = opendir(vd.c_str())) {
                while (dirent* de = readdir(dd)) {
                    const std::string nm = de->d_name;
                    if (nm != "." && nm != "..") ::unlink((vd + "/" + nm).c_str());
                }
                closedir(dd);
            }
            ::rmdir(vd.c_str());
            return DTE_OK;
        }
        std::sort(chunks.begin(), chunks.end(), [](const ChunkMeta& a, const ChunkMeta& b) {
            if (a.segment != b.segment) return a.segment < b.segment;
            return a.writer != b.writer ? a.writer < b.writer : a.first < b.first;
        });
        std::string s = "{\"format\": \"dte-delta-1\", \"version\": " + std::to_string(version) +
                        ", \"parent\": " + std::to_string(parent) + ", \"codec\": \"" + codec +
                        "\", \"writers\": " + std::to_string(nwriters) +
                        ", \"entries\": " + std::to_string(entries) + ",\n\"segments\": " +
                        segments_json(segs) + ",\n\"chunks\": [";
        for (size_t i = 0; i < chunks.size(); ++i) s += (i ? ",\n  " : "\n  ") + chunk_json(chunks[i]);
        s += "]}\n";
        if (!write_atomic(vd + "/manifest.json", s.data(), s.size())) return DTE_ERR_IO;
        const std::string latest = std::to_string(version) + "\n";
        if (!write_atomic(d + "/LATEST", latest.data(), latest.size())) return DTE_ERR_IO;
        *committed = 1;
        return DTE_OK;
    });
}

dte_status dte_store_latest(const char* dir, int64_t* version)
{
    return dte::no_throw([&]() -> dte_status {
        if (!dir || !version) return DTE_ERR_ARG;
        *version = 0;
        std::vector<uint8_t> text;
        if (!read_file(std::string(dir) + "/LATEST", text)) return DTE_OK;
        const std::string t(text.begin(), text.end());
        char* q = nullptr;
        const long long v = std::strtoll(t.c_str(), &q, 10);
        if (q == t.c_str() || v < 1) return DTE_ERR_CORRUPT;
        *version = v;
        return DTE_OK;
    });
}

dte_status dte_store_chain(const char* dir, int64_t base, int64_t latest, int64_t* out, int32_t max,
                           int32_t* n)
{
    return dte::no_throw([&]() -> dte_status {
        if (!dir || !n || base < 0 || latest < base || max < 0 || (max > 0 && !out)) return DTE_ERR_ARG;
        *n = 0;
        std::vector<int64_t> chain;
        int64_t v = latest;
        while (v != base) {
            if (v < base || v == 0) return DTE_ERR_CHAIN;
            if ((int64_t)chain.size() >= max) return DTE_ERR_ARG;
            Manifest m;
            const dte_status st = load_manifest(dir, v, m);
            if (st != DTE_OK) return st;
            chain.push_back(v);
            if (m.parent >= v) return DTE_ERR_CORRUPT;
            v = m.parent;
        }
        std::reverse(chain.begin(), chain.end());
        for (size_t i = 0; i < chain.size(); ++i) out[i] = chain[i];
        *n = (int32_t)chain.size();
        return DTE_OK;
    });
}


dte_status dte_store_read_host(const char* dir, int64_t version, int64_t base, int64_t* idx,
                               uint16_t* val, int64_t capacity, int64_t* count, int32_t threads,
                               dte_store_stats* stats)
{
    return dte::no_throw([&]() -> dte_status {
        if (!dir || version < 1 || base < 0 || capacity < 0 || (capacity > 0 && (!idx || !val)) || !count ||
            threads < 1 || threads > 64)
            return DTE_ERR_ARG;
        Manifest m;
        const dte_status st = load_manifest(dir, version, m);
        if (st != DTE_OK) return st;
        if (m.parent != base) return DTE_ERR_CHAIN;
        *count = m.entries;
        const dte_status rs = read_chunks(dir, m, threads, [&](size_t k, const uint32_t* local,
                                                               const uint16_t* v) {
            const ChunkMeta& c = m.chunks[k];
            const int64_t at = m.offset[k];
            const int64_t b = m.segs[c.segment].begin;
            for (int64_t i = 0; i < c.count && at + i < capacity; ++i) {
                idx[at + i] = b + (int64_t)local[i];
                val[at + i] = v[i];
            }
            return DTE_OK;
        });
        if (rs != DTE_OK) return rs;
        read_stats(stats, m);
        return DTE_OK;
    });
}

dte_status dte_store_read_device(const char* dir, int64_t version, int64_t base, int64_t* idx,
                                 uint16_t* val, int64_t capacity, int64_t* count, int32_t threads,
                                 dte_store_stats* stats, void* stream)
{
    return dte::no_throw([&]() -> dte_status {
        if (!dir || version < 1 || base < 0 || capacity < 0 || (capacity > 0 && (!idx || !val)) || !count ||
            threads < 1 || threads > 64)
            return DTE_ERR_ARG;
        Manifest m;
        dte_status st = load_manifest(dir, version, m);
        if (st != DTE_OK) return st;
        if (m.parent != base) return DTE_ERR_CHAIN;
        *count = m.entries;
        const int64_t n = std::min(m.entries, capacity);
        const hipStream_t s = (hipStream_t)stream;
        // chunk table: first entry and segment base of every chunk that fits
        std::vector<int64_t> first, cbase;
        for (size_t k = 0; k < m.chunks.size() && m.offset[k] < n; ++k) {
            first.push_back(m.offset[k]);
            cbase.push_back(m.segs[m.chunks[k].segment].begin);
        }
        const int32_t nchunk = (int32_t)first.size();
        int64_t biggest = 1;
        for (const ChunkMeta& c : m.chunks) biggest = std::max(biggest, c.count);
        DevBuf dlocal, dfirst, dbase;
        if (!dlocal.alloc((size_t)std::max<int64_t>(n, 1) * 4) || !dfirst.alloc(first.size() * 8) ||
            !dbase.alloc(cbase.size() * 8))
            return DTE_ERR_HIP;
        uint32_t* loc = static_cast<uint32_t*>(dlocal.p);
        Ring ring(threads + 2, biggest);
        if (!ring.ok()) return DTE_ERR_HIP;
        std::mutex copy_mutex;   // one copier at a time on the stream
        int device = 0;
        if (hipGetDevice(&device) != hipSuccess) return DTE_ERR_HIP;
        st = read_chunks(dir, m, threads, [&](size_t k, const uint32_t* local, const uint16_t* v) {
            const int64_t at = m.offset[k];
            if (at >= n) return DTE_OK;
            const int64_t c = std::min(m.chunks[k].count, n - at);
            const int slot = ring.acquire();
            std::memcpy(ring.local(slot), local, (size_t)c * 4);
            std::memcpy(ring.val(slot), v, (size_t)c * 2);
            dte_status r = DTE_OK;
            {
                std::lock_guard<std::mutex> g(copy_mutex);
                // pool threads start on device 0: use the caller's device
                if (hipSetDevice(device) != hipSuccess ||
                    hipMemcpyAsync(loc + at, ring.local(slot), (size_t)c * 4, hipMemcpyHostToDevice, s) !=
                        hipSuccess ||
                    hipMemcpyAsync(val + at, ring.val(slot), (size_t)c * 2, hipMemcpyHostToDevice, s) !=
                        hipSuccess ||
                    hipStreamSynchronize(s) != hipSuccess)
                    r = DTE_ERR_HIP;
            }
            ring.release(slot);
            return r;
        });
        if (st != DTE_OK) return st;
        if (n > 0) {
            if (hipMemcpyAsync(dfirst.p, first.data(), first.size() * 8, hipMemcpyHostToDevice, s) !=
                    hipSuccess ||
                hipMemcpyAsync(dbase.p, cbase.data(), cbase.size() * 8, hipMemcpyHostToDevice, s) != hipSuccess)
                return DTE_ERR_HIP;
            const int64_t want = (n + 255) / 256;
            const int64_t cap = (int64_t)device_cus() * 8;
            hipLaunchKernelGGL(widen_kernel, dim3((unsigned)std::min(want, cap)), dim3(256), 0, s, loc, n,
                               static_cast<const int64_t*>(dfirst.p), static_cast<const int64_t*>(dbase.p),
                               nchunk, idx);
            if (hipGetLastError() != hipSuccess) return DTE_ERR_HIP;
        }
        if (hipStreamSynchronize(s) != hipSuccess) return DTE_ERR_HIP;
        read_stats(stats, m);
        return DTE_OK;
    });
}

}  // extern "C"
