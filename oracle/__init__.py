"""fp64 CPU oracle of the per-position scoring (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline leg
import this package. The product path never does.
"""
from .olive_oracle import (REGION_ALL, REGION_STUDENT, REGION_TEACHER, kl_teacher_student,
                           log_softmax_stats, masks, project, row_scores, score)

__all__ = ["REGION_ALL", "REGION_STUDENT", "REGION_TEACHER", "kl_teacher_student",
           "log_softmax_stats", "masks", "project", "row_scores", "score"]
