/*
 * fastcall.c -- a CPython extension with one function, apply(), that passes its integer
 * arguments straight to stencil_apply: the call path of Plan.run in binding.py.
 *
 * Argument marshalling only.  Calling the entry point through ctypes converts every
 * argument on every call (about 1 us per call on the GPU hosts, against 2.5 us for the
 * library's own checks and kernel launch); this module parses ten integers and calls the
 * C function directly, with the interpreter lock released as ctypes releases it.  The
 * library is linked by name with an $ORIGIN run path, so the extension uses the
 * libstencil.so beside it.
 */
#define PY_SSIZE_T_CLEAN
#include <Python.h>

#include "stencil.h"

/* apply(plan, in, out, dims, coeffs, field, radius, boundary, steps, stream) -> status.
 * plan, in, out, dims (address of an int64_t[3]), coeffs, field and stream are addresses
 * as Python integers (0 for NULL); radius, boundary and steps are ints. */
static PyObject *fastcall_apply(PyObject *self, PyObject *const *args, Py_ssize_t nargs)
{
    (void)self;
    if (nargs != 10) {
        PyErr_SetString(PyExc_TypeError, "apply() takes exactly 10 arguments");
        return NULL;
    }
    void *p[7];
    static const int ptr_arg[7] = {0, 1, 2, 3, 4, 5, 9};
    for (int i = 0; i < 7; ++i) {
        PyObject *o = args[ptr_arg[i]];
        if (o == Py_None) {
            p[i] = NULL;
            continue;
        }
        p[i] = PyLong_AsVoidPtr(o);
        if (p[i] == NULL && PyErr_Occurred())
            return NULL;
    }
    const long radius = PyLong_AsLong(args[6]);
    const long boundary = PyLong_AsLong(args[7]);
    const long steps = PyLong_AsLong(args[8]);
    if (PyErr_Occurred())
        return NULL;
    if (radius < INT32_MIN || radius > INT32_MAX || boundary < INT32_MIN ||
        boundary > INT32_MAX || steps < INT32_MIN || steps > INT32_MAX) {
        PyErr_SetString(PyExc_OverflowError, "radius, boundary and steps must fit int32");
        return NULL;
    }
    /* the interpreter lock is released during the call, as ctypes does, so that calls
     * from several threads (on different plans) overlap */
    stencil_status st;
    Py_BEGIN_ALLOW_THREADS
    st = stencil_apply((stencil_plan_t)p[0], p[1], p[2], (const int64_t *)p[3], p[4], p[5],
                       (int32_t)radius, (int32_t)boundary, (int32_t)steps, (hipStream_t)p[6]);
    Py_END_ALLOW_THREADS
    return PyLong_FromLong((long)st);
}

static PyMethodDef fastcall_methods[] = {
    {"apply", (PyCFunction)(void (*)(void))fastcall_apply, METH_FASTCALL,
     "apply(plan, in, out, dims, coeffs, field, radius, boundary, steps, stream) -> status"},
    {NULL, NULL, 0, NULL},
};

static struct PyModuleDef fastcall_module = {
    PyModuleDef_HEAD_INIT, "_fastcall", "stencil_apply called without ctypes conversion", -1,
    fastcall_methods, NULL, NULL, NULL, NULL,
};

PyMODINIT_FUNC PyInit__fastcall(void)
{
    return PyModule_Create(&fastcall_module);
}
