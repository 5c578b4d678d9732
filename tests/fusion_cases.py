"""Programs in which a product folds into the sum or difference that reads it
(and cases where it must not): shared by the emulator and GPU tests."""
from workloads.bytecode import Asm


def fusion_programs():
    """Products folded into a sum or difference (and cases that must not be):
    (bytecode, n_params, forms that must appear)."""
    def mat(A, base):
        for i in range(4):
            A.param(base + i)
        A.pack(2, 2)
    progs = []
    progs.append((Asm(3, 0).param(0).param(1).mul().param(2).add().halt().bytes(), 3, {1}))
    progs.append((Asm(3, 0).param(0).param(1).mul().param(2).sub().halt().bytes(), 3, {30}))
    progs.append((Asm(3, 0).param(2).param(0).param(1).mul().sub().halt().bytes(), 3, {31}))
    # a product read twice is formed
    progs.append((Asm(3, 0).param(0).param(1).mul().storel(0).loadl(0).param(2).add().loadl(0).mul().halt().bytes(),
                  3, set()))
    # p0*p1 - p2*p3: one side folds
    progs.append((Asm(4, 0).param(0).param(1).mul().param(2).param(3).mul().sub().halt().bytes(), 4, {30}))
    # elementwise 2x2: A .* B + C, then trace
    A = Asm(12, 0)
    mat(A, 0), mat(A, 4)
    A.mul()
    mat(A, 8)
    A.add().trace()
    progs.append((A.halt().bytes(), 12, set()))
    # broadcast scalar * matrix + matrix: not folded (shapes differ)
    A = Asm(9, 0)
    A.param(8)
    mat(A, 0)
    A.mul()
    mat(A, 4)
    A.add().trace()
    progs.append((A.halt().bytes(), 9, set()))
    # a chain of folded products
    A = Asm(5, 0).param(0).param(1).mul().param(2).add().param(3).mul().param(4).sub()
    progs.append((A.halt().bytes(), 5, {30}))
    return progs

