"""ORACLE - test infrastructure only: the computation-distribution law.

HeteGen Sec. 3.2 "Computation Distribution": with W the module's parameters, alpha
the fraction of them processed on the GPU and V_CPU, V_GPU, V_COM the speeds of CPU
compute, GPU compute and CPU-to-GPU transfer (parameter size divided by time,
Fig. 1 caption), the balance of Eq. 4 is

    (1 - alpha) W / V_CPU  =  alpha W / V_GPU  +  alpha W / V_COM,

solved in closed form by Eq. 5:

    alpha = V_GPU V_COM / (V_CPU V_GPU + V_CPU V_COM + V_COM V_GPU),

approximated by Eq. 6 (GPU time neglected) as alpha ~ V_COM / (V_COM + V_CPU),
which Eq. 7 restates with whole-module times T' = W / V.  Sec. 4.2 (Eq. 8-9) splits
communication into pinning and transfer that run concurrently, so T_COM =
max(T_PIN, T_TRANS), i.e. V_COM = min(V_PIN, V_TRANS); with weights pinned once at
load time the pin term vanishes (a reading: the paper pins per module at run time).

The library's alpha is the CPU fraction, 1 - alpha_paper; a module kept wholly on
the GPU (Sec. 4.5, the module scheduler's placement) has CPU fraction 0.
"""
import math


def v_com(h2d_Bps, pin_Bps=0.0):
    """Effective communication speed from Eq. 8: T_COM = max(T_PIN, T_TRANS).

    pin_Bps <= 0 means the weight is already pinned (T_PIN = 0)."""
    if pin_Bps and pin_Bps > 0:
        return min(h2d_Bps, pin_Bps)
    return h2d_Bps


def alpha_gpu_eq5(V_cpu, V_gpu, V_com):
    """Eq. 5, first form, in the paper's notation (GPU fraction)."""
    return (V_gpu * V_com) / (V_cpu * V_gpu + V_cpu * V_com + V_com * V_gpu)


def alpha_gpu_eq6(V_cpu, V_com):
    """Eq. 6: GPU compute time neglected."""
    return V_com / (V_com + V_cpu)


def alpha_gpu_eq7(T_cpu_whole, T_com_whole):
    """Eq. 7 (and Eq. 9 with T_COM = max(T_PIN, T_TRANS)): whole-module times."""
    return T_cpu_whole / (T_cpu_whole + T_com_whole)


def plan_cpu_fraction(cpu_Bps, h2d_Bps, hbm_Bps, pin_Bps=0.0, resident=False, approx=False):
    """CPU fraction of one linear (library convention = 1 - alpha_paper)."""
    if resident:
        return 0.0
    Vc = v_com(h2d_Bps, pin_Bps)
    a_gpu = alpha_gpu_eq6(cpu_Bps, Vc) if approx else alpha_gpu_eq5(cpu_Bps, hbm_Bps, Vc)
    return min(1.0, max(0.0, 1.0 - a_gpu))


def balance_residual(alpha_gpu, V_cpu, V_gpu, V_com):
    """Left minus right side of Eq. 4 per unit of W (seconds per byte)."""
    return (1.0 - alpha_gpu) / V_cpu - (alpha_gpu / V_gpu + alpha_gpu / V_com)

