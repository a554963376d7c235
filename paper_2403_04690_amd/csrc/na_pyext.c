/*
 * na_pyext.c -- a CPython extension that calls na_forward / na_backward of
 * libna.so with the binding's arguments (Python ints for sizes and addresses,
 * a float for the scale), as a cheaper alternative to ctypes' conversion of
 * sixteen or twenty arguments on every call.  It only marshals: the functions
 * are passed in as addresses taken from the library the binding loaded (so
 * NA_LIBRARY keeps selecting the build), nothing is linked, and no torch type
 * is involved.  The binding falls back to ctypes when this module is absent.
 *
 *   forward(fn, rank, extents, kernel_size, dilation, causal, batch, heads,
 *           head_dim, dtype, scale, q, k, v, out, logsumexp, stream) -> status
 *   backward(fn, rank, extents, kernel_size, dilation, causal, batch, heads,
 *            head_dim, dtype, scale, q, k, v, out, logsumexp, dout, dq, dk, dv,
 *            stream) -> status
 *
 * Array arguments are the addresses of the problem's int64 / int32 arrays
 * (0 for a NULL causal array); the GIL is released for the call.
 */
#define PY_SSIZE_T_CLEAN
#include <Python.h>
#include <stdint.h>

#include "na.h"

typedef na_status (*fwd_fn)(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*,
                            int64_t, int64_t, int64_t, na_dtype, float, const void*, const void*,
                            const void*, void*, float*, na_stream_t);
typedef na_status (*bwd_fn)(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*,
                            int64_t, int64_t, int64_t, na_dtype, float, const void*, const void*,
                            const void*, const void*, const float*, const void*, void*, void*,
                            void*, na_stream_t);

/* The problem arguments shared by both calls: args[1] .. args[10]. */
typedef struct {
    int rank;
    const int64_t* extents;
    const int32_t *ks, *ds, *causal;
    int64_t batch, heads, head_dim;
    na_dtype dtype;
    float scale;
} problem_t;

static int read_problem(PyObject* const* args, problem_t* p) {
    p->rank = (int)PyLong_AsLong(args[1]);
    p->extents = (const int64_t*)PyLong_AsVoidPtr(args[2]);
    p->ks = (const int32_t*)PyLong_AsVoidPtr(args[3]);
    p->ds = (const int32_t*)PyLong_AsVoidPtr(args[4]);
    p->causal = (const int32_t*)PyLong_AsVoidPtr(args[5]);
    p->batch = (int64_t)PyLong_AsLongLong(args[6]);
    p->heads = (int64_t)PyLong_AsLongLong(args[7]);
    p->head_dim = (int64_t)PyLong_AsLongLong(args[8]);
    p->dtype = (na_dtype)PyLong_AsLong(args[9]);
    p->scale = (float)PyFloat_AsDouble(args[10]);
    return PyErr_Occurred() ? -1 : 0;
}

static int read_pointers(PyObject* const* args, Py_ssize_t first, Py_ssize_t n, void** out) {
    for (Py_ssize_t i = 0; i < n; ++i) out[i] = PyLong_AsVoidPtr(args[first + i]);
    return PyErr_Occurred() ? -1 : 0;
}

static PyObject* na_fast_forward(PyObject* self, PyObject* const* args, Py_ssize_t nargs) {
    (void)self;
    if (nargs != 17) {
        PyErr_SetString(PyExc_TypeError, "forward takes 17 arguments");
        return NULL;
    }
    fwd_fn fn = (fwd_fn)PyLong_AsVoidPtr(args[0]);
    problem_t p;
    void* ptr[6];
    if (PyErr_Occurred() || !fn || read_problem(args, &p) || read_pointers(args, 11, 6, ptr)) {
        if (!PyErr_Occurred()) PyErr_SetString(PyExc_ValueError, "NULL function");
        return NULL;
    }
    na_status st;
    Py_BEGIN_ALLOW_THREADS
    st = fn(p.rank, p.extents, p.ks, p.ds, p.causal, p.batch, p.heads, p.head_dim, p.dtype,
            p.scale, ptr[0], ptr[1], ptr[2], ptr[3], (float*)ptr[4], (na_stream_t)ptr[5]);
    Py_END_ALLOW_THREADS
    return PyLong_FromLong((long)st);
}

static PyObject* na_fast_backward(PyObject* self, PyObject* const* args, Py_ssize_t nargs) {
    (void)self;
    if (nargs != 21) {
        PyErr_SetString(PyExc_TypeError, "backward takes 21 arguments");
        return NULL;
    }
    bwd_fn fn = (bwd_fn)PyLong_AsVoidPtr(args[0]);
    problem_t p;
    void* ptr[10];
    if (PyErr_Occurred() || !fn || read_problem(args, &p) || read_pointers(args, 11, 10, ptr)) {
        if (!PyErr_Occurred()) PyErr_SetString(PyExc_ValueError, "NULL function");
        return NULL;
    }
    na_status st;
    Py_BEGIN_ALLOW_THREADS
    st = fn(p.rank, p.extents, p.ks, p.ds, p.causal, p.batch, p.heads, p.head_dim, p.dtype,
            p.scale, ptr[0], ptr[1], ptr[2], ptr[3], (const float*)ptr[4], ptr[5], ptr[6], ptr[7],
            ptr[8], (na_stream_t)ptr[9]);
    Py_END_ALLOW_THREADS
    return PyLong_FromLong((long)st);
}

static PyMethodDef methods[] = {
    {"forward", (PyCFunction)(void (*)(void))na_fast_forward, METH_FASTCALL,
     "na_forward through a function address; returns the status"},
    {"backward", (PyCFunction)(void (*)(void))na_fast_backward, METH_FASTCALL,
     "na_backward through a function address; returns the status"},
    {NULL, NULL, 0, NULL},
};

static struct PyModuleDef module = {PyModuleDef_HEAD_INIT, "_na_fast",
                                    "Argument marshalling for libna.so's hot calls", -1, methods,
                                    NULL, NULL, NULL, NULL};

PyMODINIT_FUNC PyInit__na_fast(void) { return PyModule_Create(&module); }
