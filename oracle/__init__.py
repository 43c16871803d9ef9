"""CPU oracle for the quantized conv / dense / requantize path.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark may import it; the product library never does, and the two
share no code.

* ``oracle.oracle`` -- numpy front end of the plain C int64 loop nests.
* ``oracle.exact``  -- pure-Python exact-rational reference for tiny inputs.
"""
