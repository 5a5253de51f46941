"""CPU oracle for the GPT-2 training step.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this package. The HIP library and
its Python binding never import it, and it imports nothing from them.

Every function is the plain definition of one step of the training step the
paper describes (sections "Model" and "Optimisation and precision", Figure 1),
written with numpy in the dtype of its inputs (fp32 for parity, fp64 for the
finite-difference pins). Where the paper is silent, the reading taken is named
in the docstring.
"""
from .gpt2 import *  # noqa: F401,F403
