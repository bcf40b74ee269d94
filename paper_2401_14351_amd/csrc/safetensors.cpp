// Converter front-end for safetensors checkpoints (the format Hugging Face
// models ship in), so that a framework checkpoint can be turned into the
// loading-optimized format directly (Sec. 4.1 converts checkpoints from
// various frameworks once, before serving).
//
// A safetensors shard is a u64 little-endian header length N, N bytes of
// JSON mapping each tensor name to {dtype, shape, data_offsets: [begin, end)}
// (plus an optional "__metadata__" object), then the tensors' raw bytes.
// Tensors of every shard, in shard order and within a shard in the order
// their bytes sit in the file, stream into the partition writer, so every
// shard is read front to back once.  Host-only.
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstring>
#include <string>
#include <vector>

#include "format.hpp"
#include "json.hpp"

using namespace sllm;

namespace {

constexpr uint64_t kMaxHeader = 100ull << 20;  // the format caps its JSON header at 100 MB

struct Entry {
    std::string name;
    uint32_t dtype;
    std::vector<int64_t> shape;
    uint64_t begin, end;
};

int32_t dtype_code(const std::string& s, uint32_t* out) {
    if (s == "F32") *out = SLLM_DTYPE_F32;
    else if (s == "F16") *out = SLLM_DTYPE_F16;
    else if (s == "BF16") *out = SLLM_DTYPE_BF16;
    else if (s == "I8") *out = SLLM_DTYPE_I8;
    else return SLLM_E_INVAL;
    return SLLM_OK;
}

int32_t pread_all(int fd, void* buf, uint64_t n, uint64_t off, const char* path) {
    uint8_t* p = static_cast<uint8_t*>(buf);
    while (n) {
        ssize_t r = ::pread(fd, p, n, (off_t)off);
        if (r < 0 && errno == EINTR) continue;
        if (r <= 0) return fail(SLLM_E_IO, "read %s at %llu: %s", path, (unsigned long long)off,
                                r < 0 ? std::strerror(errno) : "unexpected end of file");
        p += r;
        off += (uint64_t)r;
        n -= (uint64_t)r;
    }
    return SLLM_OK;
}

// Parse and check one shard's header; entries come back in file order.
int32_t read_header(int fd, uint64_t file_size, const char* path, uint64_t* data_start, std::vector<Entry>* out) {
    uint64_t n = 0;
    if (file_size < 8) return fail(SLLM_E_FORMAT, "%s: shorter than a safetensors header", path);
    SLLM_TRY(pread_all(fd, &n, 8, 0, path));
    if (n > kMaxHeader || n > file_size - 8) return fail(SLLM_E_FORMAT, "%s: bad header length %llu", path, (unsigned long long)n);
    std::string text(n, '\0');
    SLLM_TRY(pread_all(fd, &text[0], n, 8, path));
    json::Value root;
    json::Parser parser(text.data(), text.size());
    if (!parser.parse(&root)) return fail(SLLM_E_FORMAT, "%s: header is not JSON: %s", path, parser.error().c_str());
    if (root.kind != json::Value::Object) return fail(SLLM_E_FORMAT, "%s: header is not a JSON object", path);
    *data_start = 8 + n;
    const uint64_t data_len = file_size - 8 - n;
    out->clear();
    for (const auto& f : root.fields) {
        if (f.first == "__metadata__") continue;
        const json::Value& v = f.second;
        const json::Value* dt = v.get("dtype");
        const json::Value* sh = v.get("shape");
        const json::Value* of = v.get("data_offsets");
        if (v.kind != json::Value::Object || !dt || dt->kind != json::Value::String || !sh ||
            sh->kind != json::Value::Array || !of || of->kind != json::Value::Array || of->items.size() != 2)
            return fail(SLLM_E_FORMAT, "%s: tensor '%s' lacks dtype, shape or data_offsets", path, f.first.c_str());
        Entry e;
        e.name = f.first;
        if (dtype_code(dt->s, &e.dtype) != SLLM_OK)
            return fail(SLLM_E_INVAL, "%s: tensor '%s' has dtype %s; f32, f16, bf16 and i8 are supported", path,
                        f.first.c_str(), dt->s.c_str());
        if (sh->items.size() > SLLM_MAX_NDIM)
            return fail(SLLM_E_INVAL, "%s: tensor '%s' has %zu dimensions", path, f.first.c_str(), sh->items.size());
        for (const auto& d : sh->items) {
            if (d.kind != json::Value::Number || !d.integral || d.negative || !d.fits || d.u > (uint64_t)INT64_MAX)
                return fail(SLLM_E_FORMAT, "%s: tensor '%s' has a bad dimension", path, f.first.c_str());
            e.shape.push_back((int64_t)d.u);
        }
        for (int k = 0; k < 2; ++k) {
            const json::Value& o = of->items[k];
            if (o.kind != json::Value::Number || !o.integral || o.negative || !o.fits)
                return fail(SLLM_E_FORMAT, "%s: tensor '%s' has a bad data offset", path, f.first.c_str());
        }
        e.begin = of->items[0].u;
        e.end = of->items[1].u;
        if (e.end < e.begin || e.end > data_len)
            return fail(SLLM_E_FORMAT, "%s: tensor '%s' data [%llu, %llu) is outside the file", path, f.first.c_str(),
                        (unsigned long long)e.begin, (unsigned long long)e.end);
        if (check_tensor_meta(e.name.c_str(), e.dtype, (uint32_t)e.shape.size(), e.shape.data(), e.end - e.begin) != SLLM_OK)
            return fail(SLLM_E_FORMAT, "%s: %s", path, sllm_last_error());
        out->push_back(std::move(e));
    }
    std::stable_sort(out->begin(), out->end(), [](const Entry& a, const Entry& b) { return a.begin < b.begin; });
    for (size_t i = 1; i < out->size(); ++i)
        if ((*out)[i].begin < (*out)[i - 1].end)
            return fail(SLLM_E_FORMAT, "%s: tensors '%s' and '%s' overlap", path, (*out)[i - 1].name.c_str(),
                        (*out)[i].name.c_str());
    return SLLM_OK;
}

}  // namespace

extern "C" int32_t sllm_convert_safetensors(const char* const* paths, uint64_t n_paths, const char* out_dir,
                                            const sllm_convert_opts* opts) try {
    clear_error();
    if ((n_paths && !paths) || !out_dir) return fail(SLLM_E_INVAL, "paths and out_dir must be non-NULL");
    sllm_writer* w = nullptr;
    SLLM_TRY(sllm_writer_open(out_dir, opts, &w));
    struct Abort {  // removes the partial output unless the writer was closed
        sllm_writer*& w;
        ~Abort() {
            if (w) sllm_writer_abort(w);
        }
    } abort_guard{w};
    std::vector<uint8_t> buf;
    int32_t st = SLLM_OK;
    std::string msg;
    for (uint64_t s = 0; s < n_paths && st == SLLM_OK; ++s) {
        const char* path = paths[s];
        int fd = path ? ::open(path, O_RDONLY | O_CLOEXEC) : -1;
        if (fd < 0) {
            st = fail(path ? SLLM_E_IO : SLLM_E_INVAL, "open %s: %s", path ? path : "(null)", path ? std::strerror(errno) : "");
            break;
        }
        struct Closer {
            int fd;
            ~Closer() { ::close(fd); }
        } closer{fd};
        struct stat sb;
        std::vector<Entry> entries;
        uint64_t data_start = 0;
        if (::fstat(fd, &sb) != 0) st = fail(SLLM_E_IO, "fstat %s: %s", path, std::strerror(errno));
        if (st == SLLM_OK) st = read_header(fd, (uint64_t)sb.st_size, path, &data_start, &entries);
        for (size_t i = 0; st == SLLM_OK && i < entries.size(); ++i) {
            const Entry& e = entries[i];
            const uint64_t nbytes = e.end - e.begin;
            if (buf.size() < nbytes) buf.resize(nbytes);
            st = pread_all(fd, buf.data(), nbytes, data_start + e.begin, path);
            if (st != SLLM_OK) break;
            sllm_src_tensor t{e.name.c_str(), e.dtype, (uint32_t)e.shape.size(), e.shape.data(),
                              nbytes ? buf.data() : nullptr, nbytes};
            st = sllm_writer_add(w, &t);
        }
    }
    if (st != SLLM_OK) {
        msg = sllm_last_error();
        sllm_writer_abort(w);
        w = nullptr;
        return fail(st, "%s", msg.c_str());
    }
    sllm_writer* done = w;
    w = nullptr;
    return sllm_writer_close(done);
} SLLM_CATCH_ALL
