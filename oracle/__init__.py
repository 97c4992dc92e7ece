"""CPU oracle of the Polestar layer step (test infrastructure only).

Only the test suite, the smoke check of the package entry file and the
`cpu_baseline` leg of the benchmark may import this package.  It shares no
code with the HIP path.  `polestar_ref` is the float64 NumPy oracle; `brute`
is an independent pure-Python path for tiny inputs.
"""
