/*
 * CPython marshalling for the C ABI in fastseq_hip.h.
 *
 * Each function takes the same arguments as the C entry point of the same
 * name, with pointers and the stream passed as Python ints, and returns the
 * status (or the size) unchanged.  Nothing else happens here: no checks,
 * no torch types, no arithmetic.  It exists because ctypes spends several
 * microseconds converting a dozen arguments, which is a fifth of a decode
 * step's GPU time.
 */
#define PY_SSIZE_T_CLEAN
#include <Python.h>
#include <limits.h>
#include <string.h>

#include "fastseq_hip.h"

/* Convert args[0..n) into unsigned 64-bit values (pointers, sizes) or
 * signed ints; the format string holds one letter per argument:
 * 'p' pointer / size_t, 'i' int. */
static int unpack(PyObject *const *args, Py_ssize_t nargs, const char *fmt, unsigned long long *u, int *v) {
    Py_ssize_t n = (Py_ssize_t)strlen(fmt);
    if (nargs != n) {
        PyErr_Format(PyExc_TypeError, "expected %zd arguments, got %zd", n, nargs);
        return -1;
    }
    for (Py_ssize_t i = 0; i < n; ++i) {
        PyObject *a = args[i];
        if (fmt[i] == 'p') {
            if (a == Py_None) {
                u[i] = 0;
                continue;
            }
            u[i] = PyLong_AsUnsignedLongLong(a);
        } else {
            long x = PyLong_AsLong(a);
            if (!PyErr_Occurred() && (x < INT_MIN || x > INT_MAX))
                PyErr_SetString(PyExc_OverflowError, "int argument out of range");
            v[i] = (int)x;
        }
        if (PyErr_Occurred()) return -1;
    }
    return 0;
}

#define PTR(i) ((void *)(uintptr_t)u[i])

static PyObject *py_beam_cross_attn(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[14];
    int v[14];
    (void)self;
    if (unpack(args, nargs, "pppppiiiiiippp", u, v)) return NULL;
    int st = fs_beam_cross_attn(PTR(0), PTR(1), PTR(2), (const int32_t *)PTR(3), PTR(4), v[5], v[6], v[7],
                                v[8], v[9], v[10], PTR(11), (size_t)u[12], PTR(13));
    return PyLong_FromLong(st);
}

static PyObject *py_beam_decode_step(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[20];
    int v[20];
    (void)self;
    if (unpack(args, nargs, "pppppiiiiiipiiipippp", u, v)) return NULL;
    int st = fs_beam_decode_step(PTR(0), PTR(1), PTR(2), (const int32_t *)PTR(3), PTR(4), v[5], v[6], v[7], v[8],
                                 v[9], v[10], (const int32_t *)PTR(11), v[12], v[13], v[14], (float *)PTR(15),
                                 v[16], PTR(17), (size_t)u[18], PTR(19));
    return PyLong_FromLong(st);
}

static PyObject *py_beam_prefix_attn(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[19];
    int v[19];
    (void)self;
    if (unpack(args, nargs, "ppppppiipiiiiiippp", u, v)) return NULL;
    int st = fs_beam_prefix_attn(PTR(0), PTR(1), PTR(2), (const int32_t *)PTR(3), PTR(4), PTR(5), v[6], v[7],
                                 PTR(8), v[9], v[10], v[11], v[12], v[13], v[14], PTR(15), (size_t)u[16],
                                 PTR(17));
    return PyLong_FromLong(st);
}

static PyObject *py_ngram_block(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[8];
    int v[8];
    (void)self;
    if (unpack(args, nargs, "piiiipip", u, v)) return NULL;
    int st = fs_ngram_block((const int32_t *)PTR(0), v[1], v[2], v[3], v[4], (float *)PTR(5), v[6], PTR(7));
    return PyLong_FromLong(st);
}

static PyObject *py_beam_select(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[16];
    int v[16];
    (void)self;
    if (unpack(args, nargs, "pppiiipppiiiippp", u, v)) return NULL;
    int st = fs_beam_select((const float *)PTR(0), (const float *)PTR(1), (const int32_t *)PTR(2), v[3], v[4],
                            v[5], (float *)PTR(6), (int32_t *)PTR(7), (int32_t *)PTR(8), v[9], v[10], v[11],
                            v[12], PTR(13), (size_t)u[14], PTR(15));
    return PyLong_FromLong(st);
}

static PyObject *py_cache_reorder(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[11];
    int v[11];
    (void)self;
    if (unpack(args, nargs, "pppiiiiiiip", u, v)) return NULL;
    int st = fs_cache_reorder(PTR(0), PTR(1), (const int32_t *)PTR(2), v[3], v[4], v[5], v[6], v[7], v[8], v[9],
                              PTR(10));
    return PyLong_FromLong(st);
}

static PyObject *py_ancestry_step(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[7];
    int v[7];
    (void)self;
    if (unpack(args, nargs, "pipiiip", u, v)) return NULL;
    int st = fs_beam_ancestry_step((int32_t *)PTR(0), v[1], (const int32_t *)PTR(2), v[3], v[4], v[5], PTR(6));
    return PyLong_FromLong(st);
}

static PyObject *py_beam_prefix_attn_indirect(PyObject *self, PyObject *const *args, Py_ssize_t nargs) {
    unsigned long long u[20];
    int v[20];
    (void)self;
    if (unpack(args, nargs, "pppppppiiipiiiiiippp", u, v)) return NULL;
    int st = fs_beam_prefix_attn_indirect(PTR(0), PTR(1), PTR(2), (const int32_t *)PTR(3), PTR(4), PTR(5),
                                          (const int32_t *)PTR(6), v[7], v[8], v[9], PTR(10), v[11], v[12], v[13],
                                          v[14], v[15], v[16], PTR(17), (size_t)u[18], PTR(19));
    return PyLong_FromLong(st);
}

static PyObject *py_last_error(PyObject *self, PyObject *unused) {
    (void)self;
    (void)unused;
    return PyUnicode_FromString(fs_last_error());
}

static PyMethodDef methods[] = {
    {"fs_beam_cross_attn", (PyCFunction)(void (*)(void))py_beam_cross_attn, METH_FASTCALL,
     "fs_beam_cross_attn(q, K, V, src_len, out, B, k, H, S, D, dtype, workspace, workspace_bytes, stream)"},
    {"fs_beam_decode_step", (PyCFunction)(void (*)(void))py_beam_decode_step, METH_FASTCALL,
     "fs_beam_decode_step(q, K, V, src_len, out, B, k, H, S, D, dtype, tokens, ld_tokens, t, n, logits, vocab, "
     "workspace, workspace_bytes, stream)"},
    {"fs_beam_prefix_attn", (PyCFunction)(void (*)(void))py_beam_prefix_attn, METH_FASTCALL,
     "fs_beam_prefix_attn(q, Kp, Vp, prefix_len, Kt, Vt, T, t, out, B, k, H, N, D, dtype, workspace, "
     "workspace_bytes, stream)"},
    {"fs_ngram_block", (PyCFunction)(void (*)(void))py_ngram_block, METH_FASTCALL,
     "fs_ngram_block(tokens, ld_tokens, rows, t, n, logits, V, stream)"},
    {"fs_beam_select", (PyCFunction)(void (*)(void))py_beam_select, METH_FASTCALL,
     "fs_beam_select(logits, beam_scores, tokens, ld_tokens, t, n, out_scores, out_beam, out_token, B, k, V, c, "
     "workspace, workspace_bytes, stream)"},
    {"fs_cache_reorder", (PyCFunction)(void (*)(void))py_cache_reorder, METH_FASTCALL,
     "fs_cache_reorder(K, V, parent, B, k, H, T, t, D, dtype, stream)"},
    {"fs_beam_ancestry_step", (PyCFunction)(void (*)(void))py_ancestry_step, METH_FASTCALL,
     "fs_beam_ancestry_step(anc, ld_anc, parent, B, k, t, stream)"},
    {"fs_beam_prefix_attn_indirect", (PyCFunction)(void (*)(void))py_beam_prefix_attn_indirect, METH_FASTCALL,
     "fs_beam_prefix_attn_indirect(q, Kp, Vp, prefix_len, Kt, Vt, anc, ld_anc, T, t, out, B, k, H, N, D, dtype, "
     "workspace, workspace_bytes, stream)"},
    {"fs_last_error", py_last_error, METH_NOARGS, "fs_last_error() -> str"},
    {NULL, NULL, 0, NULL},
};

static struct PyModuleDef module = {PyModuleDef_HEAD_INIT, "_fastseq_ext",
                                    "CPython marshalling for libfastseq_hip.so", -1, methods,
                                    NULL, NULL, NULL, NULL};

PyMODINIT_FUNC PyInit__fastseq_ext(void) { return PyModule_Create(&module); }
